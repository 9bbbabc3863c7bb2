// C ABI of libdpb.so: argument validation, plan lifetime, launches.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>

#include "../../include/dpb.h"
#include "dpb_internal.hpp"

using dpb::DevPlan;

static_assert(dpb::kStdSample == DPB_STD_SAMPLE, "standardization sample size");
static_assert(dpb::kStaticScratchBytes == DPB_NOALLOC_SCRATCH_BYTES, "allocation-free encoder scratch size");
using dpb::Hierarchy;

namespace {

int pow2_at_least(int v)
{
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

int table_status(int rc) { return rc; }

// Builds the host tables and the DevPlan layout of a validated hierarchy.
dpb_status fill_plan(dpb_plan* plan, const Hierarchy& h, const uint32_t* gens, uint64_t seed)
{
    plan->h = h;
    int rc = dpb::build_masks(h.d, h.level_bits[h.levels - 1], &plan->masks_h);
    if (rc) return (dpb_status)table_status(rc);
    if (gens) {
        rc = dpb::check_generators(h, gens);
        if (rc) return (dpb_status)rc;
        size_t total = 0;
        for (int l = 1; l < h.levels; ++l) total += h.branching[l];
        plan->gens_h.assign(gens, gens + total);
    } else {
        rc = dpb::draw_generators(h, seed, &plan->gens_h);
        if (rc) return (dpb_status)rc;
    }

    DevPlan& P = plan->dev;
    P.d = h.d;
    P.dp = (h.d + dpb::kChunk - 1) / dpb::kChunk * dpb::kChunk;
    P.nchunk = P.dp / dpb::kChunk;
    P.levels = h.levels;
    P.rsd = (float)(1.0 / std::sqrt((double)h.d));
    P.k_tot = 0;
    P.kmax = 0;
    int goff = 0;
    int64_t gamma_off = 0;
    for (int l = 0; l < dpb::kMaxLevels; ++l) {
        const bool live = l < h.levels;
        P.level_bits[l] = live ? h.level_bits[l] : 0;
        P.delta[l] = live && l ? h.branching[l] : 0;
        P.active[l] = live ? h.active[l] : 0;
        P.slot_base[l] = P.k_tot;
        P.k_tot += P.active[l];
        if (P.active[l] > P.kmax) P.kmax = P.active[l];
        P.mblocks[l] = (P.delta[l] + 15) / 16;
        P.cpad[l] = l && live ? pow2_at_least(h.active[l - 1] * h.branching[l]) : 0;
        P.gens_off[l] = goff;
        goff += P.delta[l];
        P.gamma_off[l] = gamma_off;
        gamma_off += (int64_t)P.mblocks[l] * P.nchunk * 64;
    }

    // code kernels: parent columns per token, padded branching, nibble groups
    const int L = h.levels;
    int maxcpt = 1;
    int64_t gt_off = 0;
    for (int l = 0; l < dpb::kMaxLevels; ++l) {
        const bool live = l >= 1 && l < L;
        P.cpt[l] = live ? pow2_at_least(h.active[l - 1]) : 0;
        P.dpad[l] = live ? (h.branching[l] + 15) / 16 * 16 : 0;
        if (P.cpt[l] > maxcpt) maxcpt = P.cpt[l];
        P.gamma_t_off[l] = gt_off;
        if (live) gt_off += (int64_t)(P.dp / 16) * (P.dpad[l] / 16) * 64;
    }
    {
        int64_t gb = 0;
        for (int l = 0; l < dpb::kMaxLevels; ++l) {
            const bool live = l >= 1 && l < L;
            P.gpad[l] = live ? (h.branching[l] + 31) / 32 * 32 : 0;
            P.gbits_off[l] = gb;
            gb += (int64_t)P.gpad[l] * (P.nchunk | 1);   // rows at stride cws (set below)
        }
    }
    P.bwd_direct = 0;
    for (int l = 1; l < L; ++l)
        if (h.branching[l] > 64) P.bwd_direct = 1;
    P.wave_tokens = maxcpt >= 16 ? 1 : 16 / maxcpt;
    P.leaf_columns = (L >= 2 && P.cpt[L - 1] >= 4 && P.cpt[L - 1] <= 16 && h.active[L - 1] >= 2 * h.active[L - 2] &&
                      P.dpad[L - 1] == 16 && P.slot_base[L - 2] + h.active[L - 2] <= dpb::kFrMax)
                         ? 1
                         : 0;
    P.nt_groups = (h.level_bits[L - 1] + 3) / 4;
    P.cws = P.nchunk | 1;
    P.prow = P.dp / 2 + 16;
    for (int l = 0; l < dpb::kMaxLevels; ++l) {
        int sh = 0;
        while ((1 << sh) < P.cpt[l]) ++sh;
        P.cpt_shift[l] = sh;
    }
    {
        // table decode: the slots not taken by leaf columns, plus room for a few unclaimed leaves
        const int nonleaf = P.leaf_columns ? P.slot_base[L - 1] : P.k_tot;
        const int want = (nonleaf + 31) / 32 * 32;
        P.fr_cap = std::min(dpb::kFrMax, std::max(32, want));
        P.pb_bytes = (L >= 2 && h.active[L - 2] > 8) ? 2 : 1;
    }

    // generator hash tables: a collision-free hash h(x) = (x ^ (x >> r)) & (2^bits - 1)
    // of each level's generators, the smallest table (>= 2 Delta entries) that has one
    P.gtab_total = 0;
    P.gens_total = goff;
    bool hashed = true;
    for (int l = 0; l < dpb::kMaxLevels; ++l) {
        P.gtab_off[l] = P.gtab_total;
        P.gtab_bits[l] = 0;
        P.gtab_shift[l] = 0;
        if (l >= 1 && l < L) {
            const uint32_t* g = plan->gens_h.data() + P.gens_off[l];
            const int n = h.branching[l];
            int bits = 1;
            while ((1 << bits) < 2 * n) ++bits;
            bool found = false;
            std::vector<char> used;
            for (; bits <= 12 && !found; ++bits) {
                const uint32_t mask = (1u << bits) - 1u;
                for (int r = 1; r < 32 && !found; ++r) {
                    used.assign((size_t)1 << bits, 0);
                    bool ok = true;
                    for (int j = 0; j < n && ok; ++j) {
                        const uint32_t x = g[j], hs = (x ^ (x >> r)) & mask;
                        ok = !used[hs];
                        used[hs] = 1;
                    }
                    if (ok) {
                        found = true;
                        P.gtab_bits[l] = bits;
                        P.gtab_shift[l] = r;
                    }
                }
                if (found) break;
            }
            if (!found) hashed = false;
            P.gtab_total += 1 << P.gtab_bits[l];
        }
    }
    if (!hashed || P.gtab_total > 8192) P.gtab_total = 0;  // no routing: slots are decoded by table
    return DPB_OK;
}

// Generator hash tables (see DevPlan::gtab): entry h holds (g_j, j) for the
// generator that hashes to h, or (0, -1).
void build_gen_tables(const dpb_plan* plan, std::vector<uint32_t>* out)
{
    const DevPlan& P = plan->dev;
    out->assign((size_t)std::max(P.gtab_total, 1) * 2, 0);
    for (size_t i = 1; i < out->size(); i += 2) (*out)[i] = 0xFFFFFFFFu;
    if (!P.gtab_total) return;
    for (int l = 1; l < P.levels; ++l) {
        const uint32_t mask = (1u << P.gtab_bits[l]) - 1u, r = (uint32_t)P.gtab_shift[l];
        uint32_t* tab = out->data() + 2 * (size_t)P.gtab_off[l];
        for (int j = 0; j < P.delta[l]; ++j) {
            const uint32_t x = plan->gens_h[P.gens_off[l] + j], hs = (x ^ (x >> r)) & mask;
            tab[2 * hs] = x;
            tab[2 * hs + 1] = (uint32_t)j;
        }
    }
}

inline uint32_t row_parity(uint32_t m, uint32_t p) { return (uint32_t)__builtin_popcount(m & p) & 1u; }

inline uint16_t pm_one(uint32_t neg) { return neg ? 0xBF80 : 0x3F80; }  // bf16 -1 / +1

// Sign-bitmap words of index (v << 4g): bit b of word w is the sign at coordinate 32w + b.
// Groups nt_groups .. kNtGroupsPadded - 1 are zero words (index nibbles there are 0),
// so kernels may fold a fixed number of groups.
void build_nibble_tables(const dpb_plan* plan, std::vector<uint32_t>* out)
{
    const DevPlan& P = plan->dev;
    out->assign((size_t)std::max(P.nt_groups, dpb::kNtGroupsPadded) * 16 * P.nchunk, 0);
    for (int g = 0; g < P.nt_groups; ++g)
        for (uint32_t v = 0; v < 16; ++v)
            for (int w = 0; w < P.nchunk; ++w) {
                uint32_t word = 0;
                for (int b = 0; b < 32; ++b) {
                    const int iota = 32 * w + b;
                    if (iota < P.d) word |= row_parity(plan->masks_h[iota], v << (4 * g)) << b;
                }
                (*out)[((size_t)g * P.nchunk + w) * 16 + v] = word;
            }
}

// Scoring A fragments in the interleaved-halves coordinate order (see DevPlan::gamma_pair).
void build_gamma_pair(const dpb_plan* plan, std::vector<uint16_t>* out)
{
    const DevPlan& P = plan->dev;
    int64_t total = 0;
    for (int l = 1; l < P.levels; ++l) total += (int64_t)P.mblocks[l] * P.nchunk * 64 * 8;
    out->assign((size_t)total, 0);
    for (int l = 1; l < P.levels; ++l) {
        const uint32_t* g = plan->gens_h.data() + P.gens_off[l];
        for (int mb = 0; mb < P.mblocks[l]; ++mb)
            for (int c = 0; c < P.nchunk; ++c)
                for (int lane = 0; lane < 64; ++lane) {
                    const int j = 16 * mb + (lane & 15), kq = lane >> 4;
                    uint16_t* dst = out->data() + (P.gamma_off[l] + ((int64_t)mb * P.nchunk + c) * 64 + lane) * 8;
                    for (int e = 0; e < 8; ++e) {
                        const int iota = 32 * c + 4 * kq + (e >> 1) + 16 * (e & 1);
                        dst[e] = (j < P.delta[l] && iota < P.d) ? pm_one(row_parity(plan->masks_h[iota], g[j])) : 0;
                    }
                }
    }
}

// Column-decode B fragments (see DevPlan::gamma_t).
void build_gamma_t(const dpb_plan* plan, std::vector<uint16_t>* out)
{
    const DevPlan& P = plan->dev;
    int64_t total = 0;
    for (int l = 1; l < P.levels; ++l) total += (int64_t)(P.dp / 16) * (P.dpad[l] / 16) * 64 * 4;
    out->assign((size_t)total, 0);
    for (int l = 1; l < P.levels; ++l) {
        const uint32_t* g = plan->gens_h.data() + P.gens_off[l];
        const int nkb = P.dpad[l] / 16;
        for (int cb = 0; cb < P.dp / 16; ++cb)
            for (int kb = 0; kb < nkb; ++kb)
                for (int lane = 0; lane < 64; ++lane) {
                    uint16_t* dst = out->data() + (P.gamma_t_off[l] + ((int64_t)cb * nkb + kb) * 64 + lane) * 4;
                    const int iota = 16 * cb + (lane & 15);
                    for (int i = 0; i < 4; ++i) {
                        const int j = 16 * kb + 4 * (lane >> 4) + i;
                        dst[i] = (j < P.delta[l] && iota < P.d) ? pm_one(row_parity(plan->masks_h[iota], g[j])) : 0;
                    }
                }
    }
}

// Child sign patterns gamma_j = R(M g_j) (§2.2 child-scoring equation) laid
// out as MFMA A fragments: lane L of fragment (mb, c) holds generator row
// 16*mb + L%16 at coordinates 32c + 8*(L/16) + e, e = 0..7, as bf16 +-1.
void build_gamma_fragments(const dpb_plan* plan, std::vector<uint16_t>* out)
{
    const DevPlan& P = plan->dev;
    int64_t total = 0;
    for (int l = 1; l < P.levels; ++l) total += (int64_t)P.mblocks[l] * P.nchunk * 64 * 8;
    out->assign((size_t)total, 0);
    for (int l = 1; l < P.levels; ++l) {
        const uint32_t* g = plan->gens_h.data() + P.gens_off[l];
        for (int mb = 0; mb < P.mblocks[l]; ++mb)
            for (int c = 0; c < P.nchunk; ++c)
                for (int lane = 0; lane < 64; ++lane) {
                    const int j = 16 * mb + (lane & 15);
                    uint16_t* dst = out->data() + (P.gamma_off[l] + ((int64_t)mb * P.nchunk + c) * 64 + lane) * 8;
                    for (int e = 0; e < 8; ++e) {
                        const int iota = 32 * c + 8 * (lane >> 4) + e;
                        uint16_t v = 0;
                        if (j < P.delta[l] && iota < P.d)
                            v = (__builtin_popcount(plan->masks_h[iota] & g[j]) & 1) ? 0xBF80 : 0x3F80;
                        dst[e] = v;
                    }
                }
    }
}

// Generator sign bitmaps (see DevPlan::gbits).
void build_gen_bits(const dpb_plan* plan, std::vector<uint32_t>* out)
{
    const DevPlan& P = plan->dev;
    int64_t total = 0;
    for (int l = 1; l < P.levels; ++l) total += (int64_t)P.gpad[l] * P.cws;
    out->assign((size_t)std::max<int64_t>(total, 1), 0);
    for (int l = 1; l < P.levels; ++l) {
        const uint32_t* g = plan->gens_h.data() + P.gens_off[l];
        for (int j = 0; j < P.delta[l]; ++j)
            for (int c = 0; c < P.nchunk; ++c) {
                uint32_t word = 0;
                for (int b = 0; b < 32; ++b) {
                    const int iota = 32 * c + b;
                    if (iota < P.d) word |= row_parity(plan->masks_h[iota], g[j]) << b;
                }
                (*out)[P.gbits_off[l] + (int64_t)j * P.cws + c] = word;
            }
    }
}

dpb_status upload(dpb_plan* plan)
{
    DevPlan& P = plan->dev;
    std::vector<uint16_t> gamma, gamma_pair, gamma_t;
    std::vector<uint32_t> nt, gbits;
    build_gen_bits(plan, &gbits);
    std::vector<uint32_t> gtab;
    build_gen_tables(plan, &gtab);
    build_gamma_fragments(plan, &gamma);
    build_gamma_pair(plan, &gamma_pair);
    build_gamma_t(plan, &gamma_t);
    build_nibble_tables(plan, &nt);
    std::vector<uint32_t> masks_p(P.dp, 0);
    std::copy(plan->masks_h.begin(), plan->masks_h.end(), masks_p.begin());

    // one device allocation, 256-byte aligned sub-buffers
    struct Part {
        const void* src;
        size_t bytes;
        size_t off;
    };
    Part parts[] = {
        {masks_p.data(), masks_p.size() * 4, 0},
        {plan->gens_h.data(), plan->gens_h.size() * 4, 0},
        {gamma.data(), gamma.size() * 2, 0},
        {gamma_pair.data(), gamma_pair.size() * 2, 0},
        {gamma_t.data(), gamma_t.size() * 2, 0},
        {nt.data(), nt.size() * 4, 0},
        {gtab.data(), gtab.size() * 4, 0},
        {gbits.data(), gbits.size() * 4, 0},
    };
    size_t total = 0;
    for (Part& p : parts) {
        p.off = total;
        total += (std::max<size_t>(p.bytes, 16) + 255) & ~(size_t)255;
    }
    if (hipGetDevice(&plan->device) != hipSuccess) {
        (void)hipGetLastError();
        return DPB_EHIP;
    }
    void* mem = nullptr;
    if (hipMalloc(&mem, total) != hipSuccess) {
        (void)hipGetLastError();
        return DPB_ENOMEM;
    }
    plan->dev_alloc = mem;
    char* base = (char*)mem;
    hipError_t e = hipMemset(base, 0, total);
    for (const Part& p : parts)
        if (e == hipSuccess && p.bytes) e = hipMemcpy(base + p.off, p.src, p.bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return DPB_EHIP;
    }
    P.masks = (const uint32_t*)(base + parts[0].off);
    P.gens = (const uint32_t*)(base + parts[1].off);
    P.gamma = base + parts[2].off;
    P.gamma_pair = base + parts[3].off;
    P.gamma_t = base + parts[4].off;
    P.nt = (const uint32_t*)(base + parts[5].off);
    P.gtab = (const uint32_t*)(base + parts[6].off);
    P.gbits = (const uint32_t*)(base + parts[7].off);
    return DPB_OK;
}

// The encoder that runs a plan: the narrow one (a level's candidates in one
// wave's registers), the wide one (a GEMM per level and a workspace), or the
// general one; None when no encoder covers the plan for this activation type.
enum class Enc { Narrow, Wide, General, None };

Enc pick_encoder(const DevPlan& P, bool x_bf16, bool std)
{
    if (dpb::encode2_supported(P) && (!std || dpb::encode2_std_supported(P))) return Enc::Narrow;
    if (dpb::encode_wide_supported(P, x_bf16)) return Enc::Wide;
    if (dpb::general_encoder_fits(P)) return Enc::General;
    return Enc::None;
}

// A plan is accepted when some encoder takes both activation types.
bool any_encoder(const DevPlan& P)
{
    return pick_encoder(P, true, false) != Enc::None && pick_encoder(P, false, false) != Enc::None;
}

dpb_status create(dpb_plan** out, const Hierarchy& h, const uint32_t* gens, uint64_t seed)
{
    if (!out) return DPB_EINVAL;
    *out = nullptr;
    int rc = dpb::validate_hierarchy(h);
    if (rc) return (dpb_status)rc;
    dpb_plan* plan = new (std::nothrow) dpb_plan();
    if (!plan) return DPB_ENOMEM;
    dpb_status s = fill_plan(plan, h, gens, seed);
    if (s == DPB_OK && (!any_encoder(plan->dev) || !dpb::code_kernels_fit(plan->dev))) s = DPB_EUNSUPPORTED;
    if (s == DPB_OK) s = upload(plan);
    // set-up of the allocation-free encoder on this device (its scratch address)
    if (s == DPB_OK) (void)dpb::scratch_setup(plan->device);
    if (s != DPB_OK) {
        dpb_plan_destroy(plan);
        return s;
    }
    *out = plan;
    return DPB_OK;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

dpb_status check_call(const dpb_plan* plan, int64_t T)
{
    if (!plan || !plan->dev_alloc || T < 0) return DPB_EINVAL;
    if (T > ((int64_t)1 << 40)) return DPB_EUNSUPPORTED;
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) {
        (void)hipGetLastError();
        return DPB_EHIP;
    }
    return dev == plan->device ? DPB_OK : DPB_EINVAL;
}

bool dtype_ok(dpb_dtype t) { return t == DPB_F32 || t == DPB_BF16; }

dpb_status launched(hipError_t e)
{
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return DPB_EHIP;
    }
    return DPB_OK;
}

// dpb_encode, dpb_encode_std and dpb_encode_noalloc: argument checks, then
// the plan's encoder.  With `own_scratch` the wide encoder's workspace is the
// library's per-device scratch array (passes sized to it) instead of the
// caller's buffer, and nothing is allocated.
dpb_status encode_any(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const float* stats,
                      int32_t* idx, float* coef, void* workspace, size_t ws_bytes, void* stream,
                      bool own_scratch = false)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(x_dtype)) return DPB_EINVAL;
    const DevPlan& P = plan->dev;
    const bool bf = x_dtype == DPB_BF16;
    const Enc e = pick_encoder(P, bf, stats != nullptr);
    if (e == Enc::None) return DPB_EUNSUPPORTED;
    int64_t chunk = 0;
    if (own_scratch && e == Enc::Wide) {
        chunk = dpb::static_chunk_tokens(P);
        if (chunk == 0) return DPB_EUNSUPPORTED;
        workspace = dpb::scratch_setup(plan->device);
        if (!workspace) return DPB_EHIP;
        ws_bytes = dpb::kStaticScratchBytes;
    }
    if (T == 0) return DPB_OK;
    if (!x || !idx || !coef || !aligned16(x) || !aligned16(idx) || !aligned16(coef) || !aligned16(stats) ||
        !aligned16(workspace))
        return DPB_EINVAL;
    hipStream_t st = (hipStream_t)stream;
    switch (e) {
    case Enc::Narrow: return launched(dpb::launch_encode2(P, x, bf, T, stats, idx, coef, st));
    case Enc::Wide:
        if (!own_scratch && (!workspace || ws_bytes < dpb::encode_wide_workspace_bytes(P, T))) return DPB_EINVAL;
        return launched(dpb::launch_encode_wide(P, x, bf, T, stats, idx, coef, workspace, st, chunk));
    case Enc::General: return launched(dpb::launch_encode(P, x, bf, T, stats, idx, coef, st));
    default: return DPB_EUNSUPPORTED;
    }
}

}  // namespace

extern "C" {

const char* dpb_status_string(dpb_status s)
{
    switch (s) {
    case DPB_OK: return "DPB_OK";
    case DPB_EINVAL: return "DPB_EINVAL: invalid argument";
    case DPB_EUNSUPPORTED: return "DPB_EUNSUPPORTED: configuration not supported by this library";
    case DPB_EHIP: return "DPB_EHIP: HIP runtime or launch failure";
    case DPB_ENOMEM: return "DPB_ENOMEM: allocation failed";
    }
    return "DPB: unknown status";
}

dpb_status dpb_hierarchy(int d, int n_bits, int levels, int branching, int beam, int k, int* level_bits,
                         int* branching_out, int* active_out)
{
    if (!level_bits || !branching_out || !active_out) return DPB_EINVAL;
    Hierarchy h;
    int rc = dpb::hierarchy_from_terms(d, n_bits, levels, branching, beam, k, &h);
    if (rc) return (dpb_status)rc;
    for (int l = 0; l < levels; ++l) {
        level_bits[l] = h.level_bits[l];
        branching_out[l] = h.branching[l];
        active_out[l] = h.active[l];
    }
    return DPB_OK;
}

dpb_status dpb_build_tables(int d, int levels, const int* level_bits, const int* branching, uint64_t seed,
                            uint32_t* masks_out, uint32_t* gens_out)
{
    if (!level_bits || !branching || levels < 1 || levels > DPB_MAX_LEVELS || !masks_out) return DPB_EINVAL;
    Hierarchy h;
    h.d = d;
    h.levels = levels;
    for (int l = 0; l < levels; ++l) {
        h.level_bits[l] = level_bits[l];
        h.branching[l] = l ? branching[l] : 0;
        h.active[l] = 1;
    }
    if (d < 2) return DPB_EINVAL;
    for (int l = 1; l < levels; ++l) {
        if (h.level_bits[l] <= h.level_bits[l - 1] || h.branching[l] < 1) return DPB_EINVAL;
        if ((uint64_t)h.branching[l] > ((uint64_t)1 << h.level_bits[l]) - ((uint64_t)1 << h.level_bits[l - 1]))
            return DPB_EINVAL;
    }
    if (h.level_bits[0] < dpb::field_degree(d) || h.level_bits[levels - 1] > 31) return DPB_EINVAL;
    std::vector<uint32_t> m, g;
    int rc = dpb::build_masks(d, h.level_bits[levels - 1], &m);
    if (rc) return (dpb_status)rc;
    std::memcpy(masks_out, m.data(), m.size() * 4);
    if (levels > 1) {
        if (!gens_out) return DPB_EINVAL;
        dpb::draw_generators(h, seed, &g);
        std::memcpy(gens_out, g.data(), g.size() * 4);
    }
    return DPB_OK;
}

dpb_status dpb_plan_create(dpb_plan** out, int d, int n_bits, int levels, int branching, int beam, int k,
                           uint64_t seed)
{
    if (!out) return DPB_EINVAL;
    *out = nullptr;
    Hierarchy h;
    int rc = dpb::hierarchy_from_terms(d, n_bits, levels, branching, beam, k, &h);
    if (rc) return (dpb_status)rc;
    return create(out, h, nullptr, seed);
}

dpb_status dpb_plan_create_ex(dpb_plan** out, int d, int levels, const int* level_bits, const int* branching,
                              const int* active, const uint32_t* generators, uint64_t seed)
{
    if (!out) return DPB_EINVAL;
    *out = nullptr;
    if (!level_bits || !active || (levels > 1 && !branching) || levels < 1 || levels > DPB_MAX_LEVELS)
        return DPB_EINVAL;
    Hierarchy h;
    h.d = d;
    h.levels = levels;
    for (int l = 0; l < levels; ++l) {
        h.level_bits[l] = level_bits[l];
        h.branching[l] = l ? branching[l] : 0;
        h.active[l] = active[l];
    }
    return create(out, h, generators, seed);
}

void dpb_plan_destroy(dpb_plan* plan)
{
    if (!plan) return;
    if (plan->dev_alloc) {
        int cur = -1;
        (void)hipGetDevice(&cur);
        if (cur != plan->device) (void)hipSetDevice(plan->device);
        (void)hipFree(plan->dev_alloc);
        if (cur != plan->device && cur >= 0) (void)hipSetDevice(cur);
        (void)hipGetLastError();
    }
    delete plan;
}

int dpb_plan_code_width(const dpb_plan* plan) { return plan ? plan->dev.k_tot : 0; }

dpb_status dpb_plan_tables(const dpb_plan* plan, uint32_t* masks_host, uint32_t* gens_host)
{
    if (!plan || !masks_host || (!gens_host && !plan->gens_h.empty())) return DPB_EINVAL;
    std::memcpy(masks_host, plan->masks_h.data(), plan->masks_h.size() * 4);
    if (!plan->gens_h.empty()) std::memcpy(gens_host, plan->gens_h.data(), plan->gens_h.size() * 4);
    return DPB_OK;
}

dpb_status dpb_plan_describe(const dpb_plan* plan, int* d, int* levels, int* level_bits, int* branching,
                             int* active, uint32_t* masks, uint32_t* gens)
{
    if (!plan) return DPB_EINVAL;
    const Hierarchy& h = plan->h;
    if (d) *d = h.d;
    if (levels) *levels = h.levels;
    for (int l = 0; l < h.levels; ++l) {
        if (level_bits) level_bits[l] = h.level_bits[l];
        if (branching) branching[l] = h.branching[l];
        if (active) active[l] = h.active[l];
    }
    if (masks) std::memcpy(masks, plan->masks_h.data(), plan->masks_h.size() * 4);
    if (gens && !plan->gens_h.empty()) std::memcpy(gens, plan->gens_h.data(), plan->gens_h.size() * 4);
    return DPB_OK;
}

dpb_status dpb_encode(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, int32_t* idx,
                      float* coef, void* workspace, size_t ws_bytes, void* stream)
{
    return encode_any(plan, x, x_dtype, T, nullptr, idx, coef, workspace, ws_bytes, stream);
}

dpb_status dpb_forward(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const float* stats,
                       int32_t* idx, float* coef, void* y, dpb_dtype y_dtype, void* workspace, size_t ws_bytes,
                       void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(x_dtype) || !dtype_ok(y_dtype)) return DPB_EINVAL;
    const DevPlan& P = plan->dev;
    if (T > 0 && (!x || !idx || !coef || !y || !aligned16(x) || !aligned16(idx) || !aligned16(coef) || !aligned16(y) ||
                  !aligned16(stats)))
        return DPB_EINVAL;
    // the encoder, then the decode kernel on the code it wrote, on one stream
    s = encode_any(plan, x, x_dtype, T, stats, idx, coef, workspace, ws_bytes, stream);
    if (s || T == 0) return s;
    return launched(dpb::launch_decode2(P, idx, coef, T, y, y_dtype == DPB_BF16, (hipStream_t)stream));
}

dpb_status dpb_decode(const dpb_plan* plan, const int32_t* idx, const float* coef, int64_t T, void* y,
                      dpb_dtype y_dtype, void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(y_dtype)) return DPB_EINVAL;
    if (T == 0) return DPB_OK;
    if (!idx || !coef || !y || !aligned16(idx) || !aligned16(coef) || !aligned16(y)) return DPB_EINVAL;
    return launched(dpb::launch_decode2(plan->dev, idx, coef, T, y, y_dtype == DPB_BF16, (hipStream_t)stream));
}

dpb_status dpb_decode_bwd(const dpb_plan* plan, const int32_t* idx, const void* grad_y, dpb_dtype g_dtype,
                          int64_t T, float* grad_coef, void* grad_x, dpb_dtype gx_dtype, void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(g_dtype) || !dtype_ok(gx_dtype)) return DPB_EINVAL;
    if (T == 0) return DPB_OK;
    if (!idx || !grad_y || !grad_coef || !grad_x || !aligned16(idx) || !aligned16(grad_y) ||
        !aligned16(grad_coef) || !aligned16(grad_x))
        return DPB_EINVAL;
    return launched(dpb::launch_decode_bwd2(plan->dev, idx, grad_y, g_dtype == DPB_BF16, T, grad_coef, grad_x,
                                           gx_dtype == DPB_BF16, (hipStream_t)stream));
}

dpb_status dpb_decode_bwd_ex(const dpb_plan* plan, const int32_t* idx, const void* grad_y, dpb_dtype g_dtype,
                             int64_t T, const float* add_grad_coef, const void* add_grad_x, const float* stats,
                             float* grad_coef, void* grad_x, dpb_dtype gx_dtype, void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(g_dtype) || !dtype_ok(gx_dtype)) return DPB_EINVAL;
    if (T == 0) return DPB_OK;
    if (!idx || !grad_y || !grad_coef || !grad_x || !aligned16(idx) || !aligned16(grad_y) ||
        !aligned16(grad_coef) || !aligned16(grad_x) || !aligned16(add_grad_coef) || !aligned16(add_grad_x))
        return DPB_EINVAL;
    if (!aligned16(stats)) return DPB_EINVAL;
    return launched(dpb::launch_decode_bwd2(plan->dev, idx, grad_y, g_dtype == DPB_BF16, T, grad_coef, grad_x,
                                           gx_dtype == DPB_BF16, (hipStream_t)stream, add_grad_coef, add_grad_x,
                                           stats));
}

size_t dpb_encode_workspace_bytes(const dpb_plan* plan, int64_t T)
{
    // the same for either activation type, with or without statistics
    if (!plan || T <= 0) return 0;
    const DevPlan& P = plan->dev;
    bool wide = false;
    for (int b = 0; b < 2; ++b)
        for (int st = 0; st < 2; ++st) wide = wide || pick_encoder(P, b != 0, st != 0) == Enc::Wide;
    return wide ? dpb::encode_wide_workspace_bytes(P, T) : 0;
}

dpb_status dpb_encode_std(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const float* stats,
                          int32_t* idx, float* coef, void* workspace, size_t ws_bytes, void* stream)
{
    if (plan && T > 0 && !stats) return DPB_EINVAL;
    return encode_any(plan, x, x_dtype, T, stats, idx, coef, workspace, ws_bytes, stream);
}

dpb_status dpb_encode_noalloc(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T,
                              const float* stats, int32_t* idx, float* coef, void* stream)
{
    return encode_any(plan, x, x_dtype, T, stats, idx, coef, nullptr, 0, stream, true);
}

dpb_status dpb_std_init(const dpb_plan* plan, float* stats, float* m2, void* stream)
{
    dpb_status s = check_call(plan, 0);
    if (s) return s;
    if (!stats || !m2 || !aligned16(stats) || !aligned16(m2)) return DPB_EINVAL;
    return launched(dpb::launch_std_init(plan->dev, stats, m2, (hipStream_t)stream));
}

size_t dpb_std_workspace_bytes(const dpb_plan* plan)
{
    return plan ? dpb::std_workspace_bytes(plan->dev) : 0;
}

dpb_status dpb_std_update(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const int32_t* idx,
                          float momentum, float eps, float* stats, float* m2, void* workspace, size_t ws_bytes,
                          void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(x_dtype) || !(momentum >= 0.f && momentum <= 1.f) || !(eps >= 0.f)) return DPB_EINVAL;
    if (!dpb::std_supported(plan->dev)) return DPB_EUNSUPPORTED;
    if (T == 0) return DPB_OK;
    if (!x || !idx || !stats || !m2 || !workspace || !aligned16(x) || !aligned16(idx) || !aligned16(stats) ||
        !aligned16(m2) || !aligned16(workspace) || ws_bytes < dpb::std_workspace_bytes(plan->dev))
        return DPB_EINVAL;
    return launched(dpb::launch_std_update(plan->dev, x, x_dtype == DPB_BF16, T, idx, momentum, eps, stats, m2,
                                           workspace, (hipStream_t)stream));
}

dpb_status dpb_normalize(const dpb_plan* plan, const void* u, dpb_dtype u_dtype, const void* ref, dpb_dtype ref_dtype,
                         const int32_t* ref_rows, int64_t T_ref, int64_t T, void* y, dpb_dtype y_dtype, float* norms,
                         void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(u_dtype) || !dtype_ok(ref_dtype) || !dtype_ok(y_dtype) || T_ref < 0) return DPB_EINVAL;
    if (!ref_rows && T_ref != T) return DPB_EINVAL;
    if (T == 0) return DPB_OK;
    if (!u || !ref || !y || !aligned16(u) || !aligned16(ref) || !aligned16(y) || !aligned16(norms) ||
        !aligned16(ref_rows))
        return DPB_EINVAL;
    if (u == y && u_dtype != y_dtype) return DPB_EINVAL;
    return launched(dpb::launch_normalize(plan->dev.d, T, u, u_dtype == DPB_BF16, ref, ref_dtype == DPB_BF16, ref_rows,
                                          T_ref, y, y_dtype == DPB_BF16, norms, (hipStream_t)stream));
}

dpb_status dpb_normalize_bwd(const dpb_plan* plan, const void* g, dpb_dtype g_dtype, const void* u, dpb_dtype u_dtype,
                             const void* ref, dpb_dtype ref_dtype, int64_t T, void* grad_u, dpb_dtype gu_dtype,
                             void* grad_ref, dpb_dtype gr_dtype, int accumulate, void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!dtype_ok(g_dtype) || !dtype_ok(u_dtype) || !dtype_ok(ref_dtype) || !dtype_ok(gu_dtype) ||
        !dtype_ok(gr_dtype))
        return DPB_EINVAL;
    if (T == 0) return DPB_OK;
    const void* all[5] = {g, u, ref, grad_u, grad_ref};
    for (const void* p : all)
        if (!p || !aligned16(p)) return DPB_EINVAL;
    if (grad_u == grad_ref || grad_u == g || grad_u == u || grad_u == ref || grad_ref == g || grad_ref == u ||
        grad_ref == ref)
        return DPB_EINVAL;
    return launched(dpb::launch_normalize_bwd(plan->dev.d, T, g, g_dtype == DPB_BF16, u, u_dtype == DPB_BF16, ref,
                                              ref_dtype == DPB_BF16, grad_u, gu_dtype == DPB_BF16, grad_ref,
                                              gr_dtype == DPB_BF16, accumulate, (hipStream_t)stream));
}

dpb_status dpb_edit_codes(const dpb_plan* plan, const int32_t* idx, const float* coef, const int32_t* tgt_idx,
                          const float* tgt_coef, int64_t T, const int32_t* rows, const int32_t* slots,
                          const int32_t* ops, int64_t E, int32_t* out_idx, float* out_coef, void* stream)
{
    dpb_status s = check_call(plan, E);
    if (s) return s;
    if (T < 0 || (!tgt_idx) != (!tgt_coef)) return DPB_EINVAL;
    if (E == 0) return DPB_OK;
    if (!idx || !coef || !rows || !slots || !ops || !out_idx || !out_coef) return DPB_EINVAL;
    const void* all[9] = {idx, coef, tgt_idx, tgt_coef, rows, slots, ops, out_idx, out_coef};
    for (const void* p : all)
        if (!aligned16(p)) return DPB_EINVAL;
    if ((const void*)out_idx == (const void*)idx || (const void*)out_coef == (const void*)coef ||
        (tgt_idx && ((const void*)out_idx == (const void*)tgt_idx || (const void*)out_coef == (const void*)tgt_coef)))
        return DPB_EINVAL;
    return launched(dpb::launch_edit_codes(idx, coef, tgt_idx, tgt_coef, T, plan->dev.k_tot, rows, slots, ops, E,
                                           out_idx, out_coef, (hipStream_t)stream));
}

size_t dpb_variance_workspace_bytes(const dpb_plan* plan, int64_t T)
{
    if (!plan || T < 0) return 0;
    const DevPlan& P = plan->dev;
    return dpb::variance_workspace_bytes((int64_t)1 << P.level_bits[P.levels - 1],
                                         dpb::variance_small_range(P.level_bits, P.levels), T * P.k_tot);
}

dpb_status dpb_variance_loss(const dpb_plan* plan, const int32_t* idx, const float* coef, int64_t T, int n_min,
                             void* workspace, size_t ws_bytes, float* loss, float* grad_coef,
                             const float* grad_scale, void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!loss || !workspace || !aligned16(workspace) || ws_bytes < dpb_variance_workspace_bytes(plan, T))
        return DPB_EINVAL;
    if (T > 0 && (!idx || !coef || !aligned16(idx) || !aligned16(coef) || !aligned16(grad_coef))) return DPB_EINVAL;
    const DevPlan& P = plan->dev;
    const int64_t nfeat = (int64_t)1 << P.level_bits[P.levels - 1];
    const int S = dpb::variance_small_range(P.level_bits, P.levels);
    if (!dpb::variance_supported(nfeat, S, T * P.k_tot)) return DPB_EUNSUPPORTED;
    return launched(dpb::launch_variance_loss(idx, coef, T, P.k_tot, nfeat, S, n_min, workspace, loss,
                                              T > 0 ? grad_coef : nullptr, grad_scale, (hipStream_t)stream));
}

dpb_status dpb_variance_grad(const dpb_plan* plan, int64_t T, const void* workspace, size_t ws_bytes,
                             float* grad_coef, const float* grad_scale, void* stream)
{
    dpb_status s = check_call(plan, T);
    if (s) return s;
    if (!workspace || !aligned16(workspace) || ws_bytes < dpb_variance_workspace_bytes(plan, T)) return DPB_EINVAL;
    if (T == 0) return DPB_OK;
    if (!grad_coef || !aligned16(grad_coef)) return DPB_EINVAL;
    const DevPlan& P = plan->dev;
    const int64_t nfeat = (int64_t)1 << P.level_bits[P.levels - 1];
    const int S = dpb::variance_small_range(P.level_bits, P.levels);
    if (!dpb::variance_supported(nfeat, S, T * P.k_tot)) return DPB_EUNSUPPORTED;
    return launched(dpb::launch_variance_grad(T, P.k_tot, nfeat, S, const_cast<void*>(workspace), grad_coef,
                                              grad_scale, (hipStream_t)stream));
}

}  // extern "C"
