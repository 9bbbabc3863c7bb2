// Host-side construction of the DPB constant tables: the packed seed matrix
// (App. A.4), the per-level generators (§2.2) and the hierarchy mapping
// (App. G Table 6 terms).  Pure C++, no GPU.
#pragma once

#include <cstdint>
#include <vector>

namespace dpb {

struct Hierarchy {
    int d = 0;
    int levels = 0;
    int level_bits[8] = {};
    int branching[8] = {};
    int active[8] = {};
};

// Returns 0 on success, a negative dpb_status otherwise.
int hierarchy_from_terms(int d, int n_bits, int levels, int branching, int beam, int k, Hierarchy* h);
int validate_hierarchy(const Hierarchy& h);

// t = ceil(log2 d) and the modulus chosen for it.
int field_degree(int d);
uint32_t field_modulus(int t);

// Row masks M_iota for iota in [0, d); bits beyond 2t are the cubic-trace
// columns used when the index width exceeds 2t.
int build_masks(int d, int index_bits, std::vector<uint32_t>* masks);

// Generators of levels 1..L-1, level by level.
int draw_generators(const Hierarchy& h, uint64_t seed, std::vector<uint32_t>* gens);
int check_generators(const Hierarchy& h, const uint32_t* gens);

}  // namespace dpb
