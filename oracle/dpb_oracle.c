/*
 * Deep Parity Bottleneck (DPB) -- CPU ORACLE.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is a plain, slow, fp64 implementation of
 * what the paper "Scaling Interpretable Transformers with Parity Bottleneck
 * Layers" defines, written so that each step can be checked against the paper
 * by eye.  It shares no code, header, table or constant generator with the
 * HIP library; only tests, the smoke check and the benchmark's CPU-baseline leg
 * may load it.  The product path never calls it.
 *
 * Readings taken where the paper is silent:
 *   R1  indices are 0-based: phi_i = e_i for 0 <= i < d  (Eq. 2 writes i <= d).
 *   R2  bit p of an index (LSB = 0) pairs with column p of M; columns 0..t-1
 *       hold coord(xi), columns t..2t-1 hold coord(xi^-1)  (App. A.4).
 *   R3  the modulus p(z) is the irreducible polynomial of degree t with the
 *       fewest terms, ties broken by the smaller integer value; this gives the
 *       paper's z^10+z^3+1 and z^11+z^2+1 (App. A.4, irreducible-polys eq.).
 *   R4  d not a power of two: t = ceil(log2 d); coordinate 0 is the field
 *       element 0 and coordinate iota >= 1 is alpha^(iota-1), alpha the
 *       numerically smallest primitive element.
 *   R5  more index bits than 2t: column 2t+q of row iota is Tr(z^q xi_iota^3).
 *   R6  generators of level l are distinct values in [2^n_{l-1}, 2^n_l) drawn
 *       by rejection from SplitMix64 (Steele, Lea, Flood 2014), state
 *       seed ^ (l * 0x9E3779B97F4A7C15), low n_l bits of each draw (§2.2).
 *   R7  candidates reached through several (parent, generator) pairs are one
 *       candidate; if fewer than K_l exist the code is padded with (-1, 0).
 *   R8  AbsTopK key: |score| descending, then index ascending; coefficient is
 *       the signed score; level-0 coefficient is x_iota itself (Eq. 2).
 *   R9  every level is emitted, level-major, so k_tot = sum_l K_l.
 *   R10 without statistics, selection scores are the raw scores (EMA
 *       standardization at its initial state, mean 0 and std 1); with them,
 *       z = (s - mu) r, r = 1/sigma (§2.2 "Score Standardization").
 *   R11 backward: grad_coef = Phi_S^T g, grad_x = Phi_S grad_coef.
 *   R20 standardized scores: level-0 z = (x - mu) r is taken in fp32 (the
 *       precision the kernel takes it in, so both sides rank the same level-0
 *       keys), levels above in fp64; mu and r are fp32 per feature.
 *   R21 statistics sample: level 0 every token of the batch; levels >= 1 the
 *       m = min(64, T) tokens floor(j T / m), each child of an active parent
 *       once per token.
 *   R22 the moving averages are of the first two raw moments of a feature's
 *       candidate scores; sigma^2 = m2 - mu^2.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* Finite field F_{2^t} in the polynomial basis (App. A.2).            */
/* An element is a t-bit vector (xi_0..xi_{t-1}) read as               */
/* xi_0 + xi_1 z + ... + xi_{t-1} z^{t-1}.  `poly` holds all t+1        */
/* coefficients of p(z), including the z^t term.                       */
/* ------------------------------------------------------------------ */

/* Product of two field elements: carry-less polynomial product reduced
 * modulo p(z).  Written as the schoolbook sum  a * sum_i b_i z^i  where
 * each a z^i is formed by repeated multiplication by z and reduction. */
uint32_t oracle_gf_mul(uint32_t a, uint32_t b, int t, uint32_t poly)
{
    uint32_t acc = 0;
    uint32_t a_zi = a; /* a * z^i mod p, for i = 0, 1, ... */
    for (int i = 0; i < t; ++i) {
        if ((b >> i) & 1u) acc ^= a_zi;
        a_zi <<= 1;
        if ((a_zi >> t) & 1u) a_zi ^= poly; /* subtract (= add) p(z) */
    }
    return acc;
}

uint32_t oracle_gf_pow(uint32_t a, uint64_t e, int t, uint32_t poly)
{
    uint32_t result = 1;
    uint32_t base = a;
    while (e) {
        if (e & 1u) result = oracle_gf_mul(result, base, t, poly);
        base = oracle_gf_mul(base, base, t, poly);
        e >>= 1;
    }
    return result;
}

/* Inverse by exponentiation xi^{-1} = xi^{2^t - 2}, with 0^{-1} = 0
 * (App. A.3 convention; App. A.4 inverse-by-exponentiation eq.). */
uint32_t oracle_gf_inv(uint32_t a, int t, uint32_t poly)
{
    if (a == 0) return 0;
    return oracle_gf_pow(a, ((uint64_t)1 << t) - 2, t, poly);
}

/* Absolute trace Tr(y) = y + y^2 + y^4 + ... + y^{2^{t-1}} (App. A.2,
 * absolute-trace eq.).  The sum is a field element equal to 0 or 1. */
uint32_t oracle_gf_trace(uint32_t y, int t, uint32_t poly)
{
    uint32_t sum = 0;
    uint32_t term = y;
    for (int j = 0; j < t; ++j) {
        sum ^= term;
        term = oracle_gf_mul(term, term, t, poly);
    }
    return sum;
}

/* ---- binary polynomials (for choosing p(z)) ---- */
static int bpoly_degree(uint64_t a)
{
    int deg = -1;
    while (a) { ++deg; a >>= 1; }
    return deg;
}

static uint64_t bpoly_mod(uint64_t a, uint64_t b)
{
    int db = bpoly_degree(b);
    int da = bpoly_degree(a);
    while (a && da >= db) {
        a ^= b << (da - db);
        da = bpoly_degree(a);
    }
    return a;
}

/* Irreducible iff no binary polynomial of degree 1..floor(t/2) divides it. */
int oracle_poly_irreducible(uint64_t f)
{
    int t = bpoly_degree(f);
    if (t < 1) return 0;
    for (int deg = 1; deg <= t / 2; ++deg) {
        for (uint64_t g = (uint64_t)1 << deg; g < ((uint64_t)1 << (deg + 1)); ++g) {
            if (bpoly_mod(f, g) == 0) return 0;
        }
    }
    return 1;
}

static int popcount64(uint64_t v)
{
    int c = 0;
    while (v) { c += (int)(v & 1u); v >>= 1; }
    return c;
}

/* Reading R3: fewest terms first, then smallest value. */
uint32_t oracle_pick_poly(int t)
{
    if (t < 1 || t > 16) return 0;
    for (int weight = 2; weight <= t + 1; ++weight) {
        for (uint64_t f = ((uint64_t)1 << t) | 1u; f < ((uint64_t)1 << (t + 1)); f += 2) {
            if (popcount64(f) != weight) continue;
            if (oracle_poly_irreducible(f)) return (uint32_t)f;
        }
    }
    return 0;
}

/* Multiplicative order of a nonzero element, by walking its powers. */
uint32_t oracle_gf_order(uint32_t a, int t, uint32_t poly)
{
    if (a == 0) return 0;
    uint32_t x = a;
    uint32_t k = 1;
    while (x != 1) {
        x = oracle_gf_mul(x, a, t, poly);
        ++k;
        if (k > ((uint32_t)1 << t)) return 0;
    }
    return k;
}

/* Reading R4: numerically smallest element of order 2^t - 1. */
uint32_t oracle_primitive_element(int t, uint32_t poly)
{
    uint32_t full = ((uint32_t)1 << t) - 1;
    for (uint32_t a = 1; a <= full; ++a) {
        if (oracle_gf_order(a, t, poly) == full) return a;
    }
    return 0;
}

int oracle_ceil_log2(int d)
{
    int t = 0;
    while ((1 << t) < d) ++t;
    return t;
}

/* ------------------------------------------------------------------ */
/* Seed matrix M, one packed row word per coordinate (App. A.4,        */
/* parity-mask-row eq.): row iota = (coord xi_iota, coord xi_iota^-1),  */
/* plus reading R5 columns when r > 2t.  Returns t, or -1 on bad args. */
/* ------------------------------------------------------------------ */
int oracle_masks(int d, int r, uint32_t* masks)
{
    if (d < 2) return -1;
    int t = oracle_ceil_log2(d);
    if (2 * t > 31 || r > 31 || r > 3 * t) return -1;
    uint32_t poly = oracle_pick_poly(t);
    int power_of_two = (d == (1 << t));
    uint32_t alpha = power_of_two ? 0 : oracle_primitive_element(t, poly);
    uint32_t alpha_pow = 1; /* alpha^(iota-1) */
    for (int iota = 0; iota < d; ++iota) {
        uint32_t xi;
        if (power_of_two) {
            xi = (uint32_t)iota; /* coordinates = bits of iota */
        } else if (iota == 0) {
            xi = 0;
        } else {
            xi = alpha_pow;
            alpha_pow = oracle_gf_mul(alpha_pow, alpha, t, poly);
        }
        uint32_t inv = oracle_gf_inv(xi, t, poly);
        uint32_t row = xi | (inv << t);
        if (r > 2 * t) {
            uint32_t cube = oracle_gf_mul(oracle_gf_mul(xi, xi, t, poly), xi, t, poly);
            uint32_t zq = 1; /* z^q */
            for (int q = 0; q < r - 2 * t; ++q) {
                uint32_t bit = oracle_gf_trace(oracle_gf_mul(zq, cube, t, poly), t, poly);
                row |= bit << (2 * t + q);
                zq = oracle_gf_mul(zq, 2u, t, poly);
            }
        }
        masks[iota] = row;
    }
    return t;
}

/* ------------------------------------------------------------------ */
/* Hashed direction entry (§2.1 Eq. 1 with App. A.4 packed-parity eq.) */
/* and the dictionary with basis override (§2.1 Eq. 2).                */
/* ------------------------------------------------------------------ */
static int parity32(uint32_t v)
{
    return __builtin_parity(v); /* popcount(v) mod 2 */
}

double oracle_phi(int d, const uint32_t* masks, int64_t i, int iota)
{
    if (i < d) return (i == iota) ? 1.0 : 0.0;
    int bit = parity32(masks[iota] & (uint32_t)i); /* (M bits(i))_iota */
    double mag = 1.0 / sqrt((double)d);
    return bit ? -mag : mag; /* R maps 0 -> +1, 1 -> -1 */
}

/* ------------------------------------------------------------------ */
/* Generators (§2.2, reading R6).                                      */
/* ------------------------------------------------------------------ */
static uint64_t splitmix64_next(uint64_t* state)
{
    uint64_t z = (*state += 0x9E3779B97F4A7C15ull);
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

/* The first n outputs of SplitMix64 from `state` (for checking the
 * generator against its published reference outputs). */
void oracle_splitmix64(uint64_t state, int n, uint64_t* out)
{
    for (int i = 0; i < n; ++i) out[i] = splitmix64_next(&state);
}

/* gens receives sum_{l>=1} delta[l] words, level by level. */
int oracle_generators(int levels, const int* nbits, const int* delta, uint64_t seed, uint32_t* gens)
{
    int out = 0;
    for (int l = 1; l < levels; ++l) {
        uint64_t lo = (uint64_t)1 << nbits[l - 1];
        uint64_t hi = (uint64_t)1 << nbits[l];
        if ((uint64_t)delta[l] > hi - lo) return -1;
        uint64_t state = seed ^ ((uint64_t)l * 0x9E3779B97F4A7C15ull);
        int have = 0;
        while (have < delta[l]) {
            uint64_t g = splitmix64_next(&state) & (hi - 1);
            if (g < lo) continue;
            int dup = 0;
            for (int j = 0; j < have; ++j) if (gens[out + j] == (uint32_t)g) dup = 1;
            if (dup) continue;
            gens[out + have] = (uint32_t)g;
            ++have;
        }
        out += delta[l];
    }
    return out;
}

/* Configuration terms (d, n, L levels, branching b, beam B, k) to the
 * per-level table (n_l, Delta_l, K_l) of App. G Table 6.  L counts level 0;
 * n_0 = ceil(log2 d), n_{L-1} = n, evenly spaced in between (floor);
 * Delta_l = b; K_l = B below the last level and k on the last level. */
int oracle_hierarchy(int d, int n, int levels, int branching, int beam, int k,
                     int* nbits, int* delta, int* active)
{
    if (levels < 1 || d < 2) return -1;
    int n0 = oracle_ceil_log2(d);
    for (int l = 0; l < levels; ++l) {
        nbits[l] = (levels == 1) ? n0 : n0 + (l * (n - n0)) / (levels - 1);
        delta[l] = (l == 0) ? 0 : branching;
        active[l] = (l == levels - 1) ? k : beam;
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Encoder: top-down beam search (§2.2).                               */
/* ------------------------------------------------------------------ */
typedef struct {
    double score; /* signed */
    int64_t index;
} cand_t;

/* AbsTopK order (reading R8): larger |score| first, then smaller index. */
static int cand_cmp(const void* pa, const void* pb)
{
    const cand_t* a = (const cand_t*)pa;
    const cand_t* b = (const cand_t*)pb;
    double fa = fabs(a->score), fb = fabs(b->score);
    if (fa > fb) return -1;
    if (fa < fb) return 1;
    if (a->index < b->index) return -1;
    if (a->index > b->index) return 1;
    return 0;
}

static int idx_cmp(const void* pa, const void* pb)
{
    int64_t a = *(const int64_t*)pa, b = *(const int64_t*)pb;
    return (a > b) - (a < b);
}

/* <phi_c, x> as a dense dot product with phi_c built from its definition. */
static double dense_score(int d, const uint32_t* masks, int64_t c, const double* x)
{
    double s = 0.0;
    for (int iota = 0; iota < d; ++iota) s += oracle_phi(d, masks, c, iota) * x[iota];
    return s;
}

/* Scores <phi_c, x> of n features ids[0..n) against one activation row x
 * (fp64, directions from the definition), for checking a selection made
 * elsewhere against the exact scores. */
void oracle_scores(int d, const uint32_t* masks, const double* x, int64_t n, const int64_t* ids, double* out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = dense_score(d, masks, ids[i], x);
}

/* Records the selection margins used to decide which GPU/oracle
 * differences come from near-ties:  boundary = (|s|_(K) - |s|_(K+1)) / |s|_(K)
 * (infinite without a (K+1)-th candidate) and order = smallest relative gap
 * between consecutive selected scores (infinite for K <= 1). */
static void margins_of(const cand_t* sorted, int n, int K, double* boundary, double* order)
{
    *boundary = INFINITY;
    *order = INFINITY;
    int take = K < n ? K : n;
    if (n > K && K > 0) {
        double a = fabs(sorted[K - 1].score), b = fabs(sorted[K].score);
        *boundary = (a > 0.0) ? (a - b) / a : 0.0;
    }
    for (int i = 0; i + 1 < take; ++i) {
        double a = fabs(sorted[i].score), b = fabs(sorted[i + 1].score);
        double m = (a > 0.0) ? (a - b) / a : 0.0;
        if (m < *order) *order = m;
    }
}

/*
 * x: [T, d] fp64.  idx/coef: [T, k_tot] level-major.  margin/order_margin:
 * [T, levels] (may be NULL).  gens: level-by-level generator words.
 * Returns 0, or -1 on bad arguments.
 */
/* Standardized level-0 score (§2.2 "Score Standardization") of a basis
 * feature: z = (x - mu) * r with r = 1/sigma, taken in fp32 -- the precision
 * the kernel takes it in -- so that both sides select the same level-0
 * features (x is an exact fp32 value).  Without statistics, z = x. */
static double std_score0(double x, const float* mu, const float* r, int64_t c)
{
    if (!mu) return x;
    const float t = (float)x - mu[c];
    const float z = t * r[c];
    return (double)z;
}

/* Standardized score of a hashed feature, in fp64. */
static double std_score(double s, const float* mu, const float* r, int64_t c)
{
    return mu ? (s - (double)mu[c]) * (double)r[c] : s;
}

static int encode_impl(int d, const uint32_t* masks, int levels, const int* nbits, const int* active,
                       const int* delta, const uint32_t* gens, const double* x, int64_t T, const float* mu,
                       const float* r, int32_t* idx, double* coef, double* margin, double* order_margin);

int oracle_encode(int d, const uint32_t* masks, int levels, const int* nbits, const int* active,
                  const int* delta, const uint32_t* gens, const double* x, int64_t T,
                  int32_t* idx, double* coef, double* margin, double* order_margin)
{
    return encode_impl(d, masks, levels, nbits, active, delta, gens, x, T, NULL, NULL, idx, coef, margin,
                       order_margin);
}

/* The encoder on standardized scores z_c = (s_c - mu_c) r_c (§2.2 "Score
 * Standardization"): AbsTopK on |z|, and z is the coefficient passed to the
 * decoder.  mu, r: fp32 per feature, N = 2^nbits[levels-1] entries each. */
int oracle_encode_std(int d, const uint32_t* masks, int levels, const int* nbits, const int* active,
                      const int* delta, const uint32_t* gens, const double* x, int64_t T, const float* mu,
                      const float* r, int32_t* idx, double* coef, double* margin, double* order_margin)
{
    if (!mu || !r) return -1;
    return encode_impl(d, masks, levels, nbits, active, delta, gens, x, T, mu, r, idx, coef, margin,
                       order_margin);
}

static int encode_impl(int d, const uint32_t* masks, int levels, const int* nbits, const int* active,
                       const int* delta, const uint32_t* gens, const double* x, int64_t T, const float* mu,
                       const float* r, int32_t* idx, double* coef, double* margin, double* order_margin)
{
    int k_tot = 0;
    int max_cand = d;
    for (int l = 0; l < levels; ++l) {
        k_tot += active[l];
        if (l > 0 && active[l - 1] * delta[l] > max_cand) max_cand = active[l - 1] * delta[l];
    }
    if (active[0] > d) return -1;

#pragma omp parallel
    {
        cand_t* cand = (cand_t*)malloc(sizeof(cand_t) * (size_t)max_cand);
        int64_t* ids = (int64_t*)malloc(sizeof(int64_t) * (size_t)max_cand);
        int64_t* parents = (int64_t*)malloc(sizeof(int64_t) * (size_t)(max_cand + 1));
#pragma omp for schedule(dynamic, 16)
        for (int64_t tok = 0; tok < T; ++tok) {
            const double* xt = x + tok * d;
            int32_t* out_idx = idx + tok * k_tot;
            double* out_coef = coef + tok * k_tot;
            int slot = 0;
            int n_parents = 0;

            /* Level 0: basis features, score = x_iota (a coordinate read). */
            for (int iota = 0; iota < d; ++iota) {
                cand[iota].score = std_score0(xt[iota], mu, r, iota);
                cand[iota].index = iota;
            }
            qsort(cand, (size_t)d, sizeof(cand_t), cand_cmp);
            if (margin) margins_of(cand, d, active[0], &margin[tok * levels], &order_margin[tok * levels]);
            for (int i = 0; i < active[0]; ++i) {
                out_idx[slot] = (int32_t)cand[i].index;
                out_coef[slot] = cand[i].score;
                parents[n_parents++] = cand[i].index;
                ++slot;
            }

            /* Levels l >= 1: children p XOR g_j of the active parents. */
            const uint32_t* g = gens;
            for (int l = 1; l < levels; ++l) {
                int n_ids = 0;
                for (int p = 0; p < n_parents; ++p)
                    for (int j = 0; j < delta[l]; ++j) ids[n_ids++] = parents[p] ^ (int64_t)g[j];
                qsort(ids, (size_t)n_ids, sizeof(int64_t), idx_cmp);
                int n_cand = 0;
                for (int i = 0; i < n_ids; ++i) {
                    if (i > 0 && ids[i] == ids[i - 1]) continue; /* reading R7 */
                    cand[n_cand].index = ids[i];
                    cand[n_cand].score = std_score(dense_score(d, masks, ids[i], xt), mu, r, ids[i]);
                    ++n_cand;
                }
                qsort(cand, (size_t)n_cand, sizeof(cand_t), cand_cmp);
                if (margin)
                    margins_of(cand, n_cand, active[l], &margin[tok * levels + l],
                               &order_margin[tok * levels + l]);
                n_parents = 0;
                for (int i = 0; i < active[l]; ++i) {
                    if (i < n_cand) {
                        out_idx[slot] = (int32_t)cand[i].index;
                        out_coef[slot] = cand[i].score;
                        parents[n_parents++] = cand[i].index;
                    } else {
                        out_idx[slot] = -1;
                        out_coef[slot] = 0.0;
                    }
                    ++slot;
                }
                g += delta[l];
            }
        }
        free(cand);
        free(ids);
        free(parents);
    }
    return 0;
}

/* ------------------------------------------------------------------ */
/* Decoder  x_hat = sum_{i in S} a_i phi_i  (§2.1) and its backward.   */
/* Slots with index < 0 are padding and contribute nothing.            */
/* ------------------------------------------------------------------ */
void oracle_decode(int d, const uint32_t* masks, int k_tot, const int32_t* idx, const double* coef,
                   int64_t T, double* y)
{
#pragma omp parallel for schedule(static)
    for (int64_t tok = 0; tok < T; ++tok) {
        double* yt = y + tok * d;
        for (int iota = 0; iota < d; ++iota) yt[iota] = 0.0;
        for (int s = 0; s < k_tot; ++s) {
            int64_t i = idx[tok * k_tot + s];
            if (i < 0) continue;
            double a = coef[tok * k_tot + s];
            for (int iota = 0; iota < d; ++iota) yt[iota] += a * oracle_phi(d, masks, i, iota);
        }
    }
}

/* grad_coef[s] = <phi_{idx_s}, g>;  grad_x = sum_s grad_coef[s] phi_{idx_s}. */
void oracle_decode_bwd(int d, const uint32_t* masks, int k_tot, const int32_t* idx, const double* g,
                       int64_t T, double* grad_coef, double* grad_x)
{
#pragma omp parallel for schedule(static)
    for (int64_t tok = 0; tok < T; ++tok) {
        const double* gt = g + tok * d;
        double* gc = grad_coef + tok * k_tot;
        double* gx = grad_x + tok * d;
        for (int iota = 0; iota < d; ++iota) gx[iota] = 0.0;
        for (int s = 0; s < k_tot; ++s) {
            int64_t i = idx[tok * k_tot + s];
            gc[s] = 0.0;
            if (i < 0) continue;
            double acc = 0.0;
            for (int iota = 0; iota < d; ++iota) acc += oracle_phi(d, masks, i, iota) * gt[iota];
            gc[s] = acc;
        }
        for (int s = 0; s < k_tot; ++s) {
            int64_t i = idx[tok * k_tot + s];
            if (i < 0) continue;
            for (int iota = 0; iota < d; ++iota) gx[iota] += gc[s] * oracle_phi(d, masks, i, iota);
        }
    }
}

/* ------------------------------------------------------------------ */
/* Coherence spectrum S(u) = sum_iota (-1)^{popcount(M_iota & u)} for   */
/* every u in [0, 2^r):  the Walsh-Hadamard transform of the histogram  */
/* of row masks (restricted to r bits).  For u = i XOR j of two hashed  */
/* indices, <phi_i, phi_j> = S(u) / d (App. A.1 hamming-correlation eq.,*/
/* with the linearity of parity, §2.1 Eq. 4).                          */
/* ------------------------------------------------------------------ */
int oracle_walsh_spectrum(int d, const uint32_t* masks, int r, int64_t* S)
{
    if (r < 1 || r > 26) return -1;
    int64_t n = (int64_t)1 << r;
    for (int64_t u = 0; u < n; ++u) S[u] = 0;
    for (int iota = 0; iota < d; ++iota) S[masks[iota] & (uint32_t)(n - 1)] += 1;
    for (int64_t h = 1; h < n; h <<= 1) {
        for (int64_t base = 0; base < n; base += 2 * h) {
            for (int64_t u = base; u < base + h; ++u) {
                int64_t a = S[u], b = S[u + h];
                S[u] = a + b;
                S[u + h] = a - b;
            }
        }
    }
    return 0;
}

/* EMA update of the standardization statistics (§2.2 "Score
 * Standardization": an exponential moving average of each feature's mean and
 * standard deviation, taken over the tokens where the feature was a
 * candidate).  A basis feature (level 0) is a candidate at every token, so its
 * sample is the column x[:, iota] of the whole batch; a feature of level
 * l >= 1 is a candidate where it is a child p XOR g_j of an active parent p
 * (a level l-1 entry of the token's code), and its sample is taken on the
 * `sample` tokens t_j = floor(j T / m), j < m = min(sample, T) (the paper's
 * sub-samples of 64 tokens), one raw score <phi_c, x_t> per token even when
 * several parents reach it.  The moving averages are of the first two raw
 * moments (reading R22): for every feature with n >= 1 samples,
 *     mu <- (1 - beta) mu + beta * mean(s),   m2 <- (1 - beta) m2 + beta * mean(s^2),
 * and sigma^2 = m2 - mu^2 (oracle_std_r), so a feature sampled once per batch
 * still estimates its spread over the batches.  Features with no sample keep
 * their state.  mu, m2: fp64 [N]. */
void oracle_std_update(int d, const uint32_t* masks, int levels, const int* nbits, const int* active,
                       const int* delta, const uint32_t* gens, const double* x, int64_t T, const int32_t* idx,
                       int sample, double beta, double* mu, double* m2)
{
    const int64_t N = (int64_t)1 << nbits[levels - 1];
    int k_tot = 0, max_ids = 1;
    for (int l = 0; l < levels; ++l) {
        k_tot += active[l];
        if (l > 0 && active[l - 1] * delta[l] > max_ids) max_ids = active[l - 1] * delta[l];
    }
    double* cnt = (double*)calloc((size_t)N, sizeof(double));
    double* s1 = (double*)calloc((size_t)N, sizeof(double));
    double* s2 = (double*)calloc((size_t)N, sizeof(double));
    int64_t* ids = (int64_t*)malloc(sizeof(int64_t) * (size_t)max_ids);
    const int64_t m = T < sample ? T : sample;
    for (int64_t t = 0; t < T; ++t)
        for (int iota = 0; iota < d; ++iota) {
            const double v = x[t * d + iota];
            cnt[iota] += 1.0;
            s1[iota] += v;
            s2[iota] += v * v;
        }
    for (int64_t j = 0; j < m; ++j) {
        const int64_t t = (j * T) / m;
        const int32_t* code = idx + t * k_tot;
        const uint32_t* g = gens;
        int slot = 0;
        for (int l = 1; l < levels; ++l) {
            const int pb = slot;          /* the parents: level l-1 entries */
            slot += active[l - 1];
            int n_ids = 0;
            for (int q = pb; q < slot; ++q) {
                if (code[q] < 0) continue;
                for (int jj = 0; jj < delta[l]; ++jj) ids[n_ids++] = (int64_t)code[q] ^ (int64_t)g[jj];
            }
            qsort(ids, (size_t)n_ids, sizeof(int64_t), idx_cmp);
            for (int i = 0; i < n_ids; ++i) {
                if (i > 0 && ids[i] == ids[i - 1]) continue;
                const int64_t c = ids[i];
                const double v = dense_score(d, masks, c, x + t * d);
                cnt[c] += 1.0;
                s1[c] += v;
                s2[c] += v * v;
            }
            g += delta[l];
        }
    }
    for (int64_t c = 0; c < N; ++c) {
        if (cnt[c] == 0.0) continue;
        mu[c] = (1.0 - beta) * mu[c] + beta * (s1[c] / cnt[c]);
        m2[c] = (1.0 - beta) * m2[c] + beta * (s2[c] / cnt[c]);
    }
    free(cnt);
    free(s1);
    free(s2);
    free(ids);
}

/* r = 1 / sigma = 1 / sqrt(max(m2 - mu^2, 0) + eps) of each of the n features
 * (the variance implied by the two moving moments, clamped at 0 against
 * rounding). */
void oracle_std_r(int64_t n, const double* mu, const double* m2, double eps, double* r)
{
    for (int64_t c = 0; c < n; ++c) {
        double v = m2[c] - mu[c] * mu[c];
        if (v < 0.0) v = 0.0;
        r[c] = 1.0 / sqrt(v + eps);
    }
}

/* ------------------------------------------------------------------ */
/* Normalized reconstruction (§2.2 "Normalized Reconstruction"): the    */
/* decoder output u of each row is rescaled to the norm of the          */
/* bottleneck input ref of that row,  y = u ||ref|| / ||u||  (y = 0 when */
/* ||u|| = 0).  norms[t] = (||ref_t||, ||u_t||).                         */
/* ------------------------------------------------------------------ */
void oracle_normalize(int d, int64_t T, const double* u, const double* ref, double* y, double* norms)
{
    for (int64_t t = 0; t < T; ++t) {
        double su = 0.0, sr = 0.0;
        for (int i = 0; i < d; ++i) {
            su += u[t * d + i] * u[t * d + i];
            sr += ref[t * d + i] * ref[t * d + i];
        }
        const double nu = sqrt(su), nr = sqrt(sr);
        norms[2 * t] = nr;
        norms[2 * t + 1] = nu;
        for (int i = 0; i < d; ++i) y[t * d + i] = nu > 0.0 ? u[t * d + i] * (nr / nu) : 0.0;
    }
}

/* Backward of the row normalization for dL/dy = g:
 *   dL/du   = (||ref|| / ||u||) (g - (<g, u> / ||u||^2) u)
 *   dL/dref = (<g, u> / (||u|| ||ref||)) ref
 * both 0 where ||u|| = 0, and dL/dref = 0 where ||ref|| = 0. */
void oracle_normalize_bwd(int d, int64_t T, const double* g, const double* u, const double* ref, double* gu,
                          double* gref)
{
    for (int64_t t = 0; t < T; ++t) {
        double su = 0.0, sr = 0.0, gdu = 0.0;
        for (int i = 0; i < d; ++i) {
            su += u[t * d + i] * u[t * d + i];
            sr += ref[t * d + i] * ref[t * d + i];
            gdu += g[t * d + i] * u[t * d + i];
        }
        const double nu = sqrt(su), nr = sqrt(sr);
        for (int i = 0; i < d; ++i) {
            gu[t * d + i] = nu > 0.0 ? (nr / nu) * (g[t * d + i] - (gdu / su) * u[t * d + i]) : 0.0;
            gref[t * d + i] = (nu > 0.0 && nr > 0.0) ? gdu / (nu * nr) * ref[t * d + i] : 0.0;
        }
    }
}

/* Code edits of the greedy feature editing (App. C.3): a source code and a
 * target code of the same shape; each edit names a source row, a slot
 * position (level and rank within the level, i.e. a column of the code) and
 * an operation, and yields one output row: the source row with that one slot
 * changed.  op 0 (zero) sets the slot's coefficient to 0; op 1 (replace)
 * takes both index and coefficient from the target at the same position;
 * op 2 (rescale) keeps the index and takes the target's coefficient; op 3
 * changes nothing.  An edit whose row, slot or op is out of range yields an
 * all-padding row (index -1, coefficient 0). */
void oracle_edit_codes(int64_t T, int k, const int32_t* idx, const double* coef, const int32_t* tidx,
                       const double* tcoef, int64_t E, const int32_t* rows, const int32_t* slots, const int32_t* ops,
                       int32_t* out_idx, double* out_coef)
{
    for (int64_t e = 0; e < E; ++e) {
        const int64_t r = rows[e];
        const int p = slots[e], op = ops[e];
        const int ok = r >= 0 && r < T && p >= 0 && p < k && op >= 0 && op <= 3;
        for (int s = 0; s < k; ++s) {
            int32_t i = ok ? idx[r * k + s] : -1;
            double c = ok ? coef[r * k + s] : 0.0;
            if (ok && s == p) {
                if (op == 0) c = 0.0;
                else if (op == 1) {
                    i = tidx[r * k + s];
                    c = tcoef[r * k + s];
                } else if (op == 2) c = tcoef[r * k + s];
            }
            out_idx[e * k + s] = i;
            out_coef[e * k + s] = c;
        }
    }
}

/* Variance auxiliary loss (§2.2 "Auxillary losses" equation): for each
 * feature i, the coefficients a_i^(t) of the slots holding i across the
 * batch form a sample; F = features with at least n_min samples;
 *     L = -(1/|F|) sum_{i in F} Var_i,   Var_i = mean(a^2) - mean(a)^2,
 * and L = 0 when F is empty.  grad[s] = dL/dcoef[s]
 *     = -(2 / |F|) (a_s - mean_i) / count_i   for the slots of i in F, else 0.
 * Padding slots (index < 0) are not samples. */
typedef struct {
    int32_t i;
    int64_t s;
} oracle_slot;

static int slot_cmp(const void* a, const void* b)
{
    const oracle_slot* x = (const oracle_slot*)a;
    const oracle_slot* y = (const oracle_slot*)b;
    if (x->i != y->i) return x->i < y->i ? -1 : 1;
    return x->s < y->s ? -1 : (x->s > y->s);
}

double oracle_variance_loss(int64_t T, int k, const int32_t* idx, const double* coef, int n_min, double* grad)
{
    const int64_t n = T * (int64_t)k;
    oracle_slot* v = (oracle_slot*)malloc((size_t)(n > 0 ? n : 1) * sizeof(oracle_slot));
    int64_t m = 0;
    for (int64_t s = 0; s < n; ++s) {
        grad[s] = 0.0;
        if (idx[s] >= 0) {
            v[m].i = idx[s];
            v[m].s = s;
            ++m;
        }
    }
    qsort(v, (size_t)m, sizeof(oracle_slot), slot_cmp);
    /* pass 1: |F|;  pass 2: sum of variances and gradients */
    int64_t nF = 0;
    for (int64_t a = 0; a < m;) {
        int64_t b = a;
        while (b < m && v[b].i == v[a].i) ++b;
        if (b - a >= n_min) ++nF;
        a = b;
    }
    double total = 0.0;
    for (int64_t a = 0; a < m;) {
        int64_t b = a;
        while (b < m && v[b].i == v[a].i) ++b;
        const int64_t c = b - a;
        if (c >= n_min && nF > 0) {
            double s1 = 0.0, s2 = 0.0;
            for (int64_t q = a; q < b; ++q) {
                s1 += coef[v[q].s];
                s2 += coef[v[q].s] * coef[v[q].s];
            }
            const double mean = s1 / (double)c;
            total += s2 / (double)c - mean * mean;
            for (int64_t q = a; q < b; ++q)
                grad[v[q].s] = -2.0 / (double)nF * (coef[v[q].s] - mean) / (double)c;
        }
        a = b;
    }
    free(v);
    return nF > 0 ? -total / (double)nF : 0.0;
}

/* Threads the OpenMP loops above use (reported next to timings). */
#include <omp.h>
int oracle_num_threads(void)
{
    return omp_get_max_threads();
}
