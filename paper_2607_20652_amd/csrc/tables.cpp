// Host-side construction of the DPB constant tables.
//
// Field arithmetic uses discrete-log tables with respect to a primitive
// element; irreducibility of the modulus is decided with Rabin's test.
#include "tables.hpp"

#include <algorithm>
#include <set>

#include "../../include/dpb.h"

namespace dpb {
namespace {

// ---------- binary polynomials over F_2 (bit q = coefficient of z^q) ----------
int pdeg(uint64_t a) { return a ? 63 - __builtin_clzll(a) : -1; }

uint64_t pmod(uint64_t a, uint64_t f)
{
    const int df = pdeg(f);
    for (int da = pdeg(a); da >= df; da = pdeg(a)) a ^= f << (da - df);
    return a;
}

// (a * b) mod f for deg a, deg b < deg f <= 31.
uint64_t pmulmod(uint64_t a, uint64_t b, uint64_t f)
{
    uint64_t prod = 0;
    for (int i = 0; b >> i; ++i)
        if ((b >> i) & 1u) prod ^= a << i;
    return pmod(prod, f);
}

uint64_t pgcd(uint64_t a, uint64_t b)
{
    while (b) {
        uint64_t r = pmod(a, b);
        a = b;
        b = r;
    }
    return a;
}

// z^(2^k) mod f by k squarings.
uint64_t frobenius_of_z(int k, uint64_t f)
{
    uint64_t x = pmod(2u, f);
    for (int i = 0; i < k; ++i) x = pmulmod(x, x, f);
    return x;
}

// Rabin: f of degree t is irreducible iff z^(2^t) = z (mod f) and, for every
// prime q dividing t, gcd(z^(2^(t/q)) - z, f) = 1.
bool rabin_irreducible(uint64_t f)
{
    const int t = pdeg(f);
    if (t < 1) return false;
    if (frobenius_of_z(t, f) != pmod(2u, f)) return false;
    for (int q = 2; q <= t; ++q) {
        bool prime = true;
        for (int e = 2; e * e <= q; ++e)
            if (q % e == 0) prime = false;
        if (!prime || t % q) continue;
        uint64_t h = frobenius_of_z(t / q, f) ^ pmod(2u, f);
        if (pdeg(pgcd(f, h)) != 0) return false;
    }
    return true;
}

// ---------- F_{2^t} through log / antilog tables ----------
struct Field {
    int t = 0;
    uint32_t order = 0;  // 2^t - 1
    uint32_t modulus = 0;
    uint32_t generator = 0;           // smallest primitive element
    std::vector<uint32_t> exp;        // exp[k] = g^k, k in [0, 2*order)
    std::vector<int32_t> log;         // log[a] for a != 0

    uint32_t mul(uint32_t a, uint32_t b) const
    {
        if (!a || !b) return 0;
        return exp[(uint32_t)log[a] + (uint32_t)log[b]];
    }
    uint32_t inv(uint32_t a) const
    {
        if (!a) return 0;  // convention 0^{-1} = 0
        return exp[(order - (uint32_t)log[a]) % order];
    }
    uint32_t trace(uint32_t y) const
    {
        if (!y) return 0;
        uint32_t acc = 0;
        uint64_t k = (uint32_t)log[y];
        for (int j = 0; j < t; ++j) {  // y^(2^j) = g^(log y * 2^j)
            acc ^= exp[k % order];
            k = (k * 2) % order;
        }
        return acc;
    }
};

bool is_primitive(uint32_t a, int t, uint32_t modulus)
{
    const uint64_t order = ((uint64_t)1 << t) - 1;
    if (order == 1) return a == 1;
    uint64_t m = order;
    for (uint64_t q = 2; q * q <= m || m > 1; ++q) {
        if (q * q > m) q = m;  // remaining factor is prime
        if (m % q) continue;
        while (m % q == 0) m /= q;
        // a^((2^t - 1)/q) must differ from 1
        uint64_t e = order / q, r = 1, base = a;
        while (e) {
            if (e & 1u) r = pmulmod(r, base, modulus);
            base = pmulmod(base, base, modulus);
            e >>= 1;
        }
        if (r == 1) return false;
    }
    return true;
}

Field make_field(int t)
{
    Field F;
    F.t = t;
    F.order = ((uint32_t)1 << t) - 1;
    F.modulus = field_modulus(t);
    for (uint32_t a = 1; a <= F.order; ++a)
        if (is_primitive(a, t, F.modulus)) {
            F.generator = a;
            break;
        }
    F.exp.assign(2 * (size_t)F.order + 1, 0);
    F.log.assign((size_t)1 << t, -1);
    uint64_t x = 1;
    for (uint32_t k = 0; k < 2 * F.order + 1; ++k) {
        F.exp[k] = (uint32_t)x;
        if (k < F.order) F.log[x] = (int32_t)k;
        x = pmulmod(x, F.generator, F.modulus);
    }
    return F;
}

uint64_t splitmix64(uint64_t* s)
{
    uint64_t z = (*s += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

}  // namespace

int field_degree(int d)
{
    int t = 0;
    while (((int64_t)1 << t) < d) ++t;
    return t;
}

// Fewest nonzero terms first, then the smallest value among them.
uint32_t field_modulus(int t)
{
    if (t < 1 || t > 16) return 0;
    for (int terms = 2; terms <= t + 1; ++terms)
        for (uint64_t f = ((uint64_t)1 << t) | 1u; f < ((uint64_t)1 << (t + 1)); f += 2)
            if (__builtin_popcountll(f) == terms && rabin_irreducible(f)) return (uint32_t)f;
    return 0;
}

int hierarchy_from_terms(int d, int n_bits, int levels, int branching, int beam, int k, Hierarchy* h)
{
    if (!h || d < 2 || levels < 1 || levels > DPB_MAX_LEVELS) return DPB_EINVAL;
    const int n0 = field_degree(d);
    h->d = d;
    h->levels = levels;
    for (int l = 0; l < levels; ++l) {
        h->level_bits[l] = levels == 1 ? n0 : n0 + (l * (n_bits - n0)) / (levels - 1);
        h->branching[l] = l ? branching : 0;
        h->active[l] = l + 1 == levels ? k : beam;
    }
    return validate_hierarchy(*h);
}

int validate_hierarchy(const Hierarchy& h)
{
    if (h.d < 2 || h.d > 4096) return h.d < 2 ? DPB_EINVAL : DPB_EUNSUPPORTED;
    if (h.levels < 1 || h.levels > DPB_MAX_LEVELS) return DPB_EINVAL;
    const int t = field_degree(h.d);
    if (h.level_bits[0] < t) return DPB_EINVAL;
    if (h.active[0] < 1 || h.active[0] > h.d) return DPB_EINVAL;
    int k_tot = h.active[0];
    for (int l = 1; l < h.levels; ++l) {
        if (h.level_bits[l] <= h.level_bits[l - 1]) return DPB_EINVAL;
        if (h.branching[l] < 1 || h.active[l] < 1) return DPB_EINVAL;
        const uint64_t level_size = ((uint64_t)1 << h.level_bits[l]) - ((uint64_t)1 << h.level_bits[l - 1]);
        if ((uint64_t)h.branching[l] > level_size) return DPB_EINVAL;
        if ((int64_t)h.active[l] > (int64_t)h.active[l - 1] * h.branching[l]) return DPB_EINVAL;
        k_tot += h.active[l];
    }
    const int n = h.level_bits[h.levels - 1];
    if (n > 30) return DPB_EINVAL;
    if (n > 3 * t || 2 * t > 31) return DPB_EUNSUPPORTED;
    for (int l = 0; l < h.levels; ++l)
        if (h.active[l] > 256) return DPB_EUNSUPPORTED;
    for (int l = 1; l < h.levels; ++l)
        if (h.branching[l] > 4096 || h.active[l - 1] * h.branching[l] > 8192) return DPB_EUNSUPPORTED;
    if (k_tot > 1024) return DPB_EUNSUPPORTED;
    return DPB_OK;
}

int build_masks(int d, int index_bits, std::vector<uint32_t>* masks)
{
    const int t = field_degree(d);
    if (t < 1 || 2 * t > 31 || index_bits > 3 * t || index_bits > 31) return DPB_EUNSUPPORTED;
    const Field F = make_field(t);
    const bool power_of_two = (1 << t) == d;
    masks->assign(d, 0);
    for (int iota = 0; iota < d; ++iota) {
        // coordinate -> field element: bits of iota when d = 2^t, otherwise
        // 0 followed by the powers g^0, g^1, ... of the primitive element.
        const uint32_t xi = power_of_two ? (uint32_t)iota : (iota == 0 ? 0u : F.exp[iota - 1]);
        uint32_t row = xi | (F.inv(xi) << t);
        for (int q = 0; 2 * t + q < index_bits; ++q) {
            const uint32_t cube = F.mul(F.mul(xi, xi), xi);
            const uint32_t zq = (uint32_t)pmod((uint64_t)1 << q, F.modulus);
            row |= F.trace(F.mul(zq, cube)) << (2 * t + q);
        }
        (*masks)[iota] = row;
    }
    return DPB_OK;
}

int draw_generators(const Hierarchy& h, uint64_t seed, std::vector<uint32_t>* gens)
{
    gens->clear();
    for (int l = 1; l < h.levels; ++l) {
        const uint64_t lo = (uint64_t)1 << h.level_bits[l - 1];
        const uint64_t mask = ((uint64_t)1 << h.level_bits[l]) - 1;
        uint64_t state = seed ^ ((uint64_t)l * 0x9E3779B97F4A7C15ull);
        std::set<uint32_t> seen;
        while ((int)seen.size() < h.branching[l]) {
            const uint64_t g = splitmix64(&state) & mask;
            if (g < lo || seen.count((uint32_t)g)) continue;
            seen.insert((uint32_t)g);
            gens->push_back((uint32_t)g);
        }
    }
    return DPB_OK;
}

int check_generators(const Hierarchy& h, const uint32_t* gens)
{
    size_t off = 0;
    for (int l = 1; l < h.levels; ++l) {
        std::set<uint32_t> seen;
        for (int j = 0; j < h.branching[l]; ++j) {
            const uint64_t g = gens[off + j];
            if (g < ((uint64_t)1 << h.level_bits[l - 1]) || g >= ((uint64_t)1 << h.level_bits[l])) return DPB_EINVAL;
            if (!seen.insert((uint32_t)g).second) return DPB_EINVAL;
        }
        off += h.branching[l];
    }
    return DPB_OK;
}

}  // namespace dpb
