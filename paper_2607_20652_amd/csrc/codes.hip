// Decode and decode-backward for gfx950.
//
// A code slot c of level l >= 1 is a child p XOR g_j of some parent p in the
// previous level, and its direction factorises as phi~_c = phi~_p (.) gamma_j
// (§2.2 factorization equation).  Both kernels first *route* every slot to a
// parent slot of the previous level and a generator j (any code may be
// passed; a slot that routes nowhere is simply handled directly).  Then:
//
//  * decode, last level: the slots routed to the same parent p form a column
//    alpha_p[j]; sum_j alpha_p[j] gamma_j = Gamma^T alpha_p runs on the matrix
//    cores (16x16x16 bf16, coefficients split exactly into bf16 terms), and
//    each column is modulated once by the parent's signs.  Other slots are
//    added directly: +-coef per coordinate, the sign being parity(M & c).
//  * backward, last level: grad_coef of the children of a parent p is
//    Gamma_l (phi~_p (.) g) -- the encoder's child-scoring contraction with g
//    in place of x (§2.2 child-scoring equation) -- on the matrix cores; the
//    parent's sign pattern comes from nibble tables (parity is linear in the
//    index bits).  The other levels select few of their parents' children
//    (K_l of K_{l-1} Delta_l), so their slots are reduced directly, one lane
//    per slot with two-element dot products.  grad_x is the decode of
//    grad_coef.
//
// Workgroups hold kCodeWaves independent waves; each wave takes groups of
// `wave_tokens` tokens in a grid-stride loop and synchronises only with itself.
// Hot loops keep their operands in registers: slot data is broadcast with
// readlane, and matrix-core fragments are fetched in batches.
#include <algorithm>

#include "scoring.hpp"

namespace dpb {
namespace {

constexpr int kThreads = 64 * kCodeWaves;
constexpr int kBatch = 16;    // leaf columns decoded per batch
constexpr int kBwdBatch = 4;
constexpr int kDecodeUnroll = 4;  // coordinates of the table decode whose reads are issued together

struct Wave {
    int lane;
    int64_t t0;
    int ntok;
    int32_t* idx;     // [TPW][k]
    float* coef;      // [TPW][k]
    int32_t* route;   // [TPW][k]: (parent slot << 16) | j (| kClaimed when decoded by its column), or -1
    int32_t* par;     // [16] parent index of each column row
    float* alpha;     // [16][dpad] column coefficients
    int32_t* claim;   // [16][dpad] lowest slot claiming (row, j)
    int32_t* fri;     // [fr_cap] indices of the table-decoded slots
    float* frc;       // [fr_cap] their coefficients (0 for basis and padding slots)
    uint32_t* frv;    // [fr_cap / 32][8][16] slot-parity tables (256-byte aligned)
    float* frt;       // [fr_cap / 4][16] signed coefficient sums
    void* pb;         // [TPW][dp] sign bits of the leaf level's parents (pb_bytes each)
    float* y;         // [TPW][dp] output accumulator (fp32)
    uint32_t* pairs;  // [TPW][prow] g as signed bf16 pairs, interleaved halves
    float* gf;        // [TPW][dp] fp32 g (fp32 activations)
    uint32_t* cw;     // [16][cws] column sign bitmaps
    float* score;     // [16][16] scores of one column block and generator tile
    const uint32_t* mask;  // [dp] row masks (shared)
    const uint32_t* gtab;  // generator hash tables (shared): (g_j, j) pairs
    const uint32_t* gens;  // generators (shared)
};

__device__ __forceinline__ int rdlane(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

typedef __attribute__((address_space(3))) uint32_t lds_u32;
typedef __attribute__((address_space(3))) float lds_f32;
__device__ __forceinline__ uint32_t lds_addr(const void* p)
{
    return (uint32_t)(size_t)(const __attribute__((address_space(3))) void*)p;
}
__device__ __forceinline__ uint32_t lds_ld(uint32_t a) { return *(const lds_u32*)(size_t)a; }
__device__ __forceinline__ float lds_ldf(uint32_t a) { return *(const lds_f32*)(size_t)a; }

// Routes every hashed slot of the last level: finds the first parent slot q
// of the previous level (in slot order) and the generator j with
// c = parent_q XOR g_j, by looking c XOR parent_q up in the level's
// collision-free generator hash: one probe per parent, all parents tried,
// four probes at a time (the reads of a batch are in flight together; the
// parents' reads, then the table's).  W.route[tt][s] = (q << 16) | j, or -1
// when no pair exists.
__device__ void route_slots(const DevPlan& P, const Wave& W)
{
    const int k = P.k_tot, l = P.levels - 1;
    if (P.gtab_total <= 0 || l < 1) return;
    const int Kp = P.active[l - 1], r = P.gtab_shift[l], sb = P.slot_base[l], sbp = P.slot_base[l - 1], d = P.d;
    const uint32_t hmask = (1u << P.gtab_bits[l]) - 1u;
    const u32x2* tab = (const u32x2*)W.gtab + P.gtab_off[l];
    for (int tt = 0; tt < W.ntok; ++tt) {
        const int32_t* parents = W.idx + tt * k + sbp;
        for (int s = sb + W.lane; s < k; s += 64) {
            int rt = -1;
            const int32_t c = W.idx[tt * k + s];
            if (c >= d) {
                for (int q0 = Kp - 1; q0 >= 0; q0 -= 4) {
                    int32_t pq[4];
                    uint32_t x[4];
                    u32x2 e[4];
#pragma unroll
                    for (int u = 0; u < 4; ++u) pq[u] = parents[max(q0 - u, 0)];
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        x[u] = (uint32_t)c ^ (uint32_t)pq[u];
                        e[u] = tab[(x[u] ^ (x[u] >> r)) & hmask];
                    }
                    // descending q: the lowest matching parent slot is kept
#pragma unroll
                    for (int u = 0; u < 4; ++u)
                        if (q0 - u >= 0 && pq[u] >= 0 && x[u] != 0u && e[u].x == x[u]) rt = ((q0 - u) << 16) | (int)e[u].y;
                }
            }
            W.route[tt * k + s] = rt;
        }
    }
}

// Bit transpose inside each 32-lane half: lane s of a half holds x_s on
// entry; on exit lane b holds the word whose bit s is bit b of x_s.  The five
// exchanges run on the vector ALU (a chain of LDS-path swizzles was slower).
__device__ __forceinline__ uint32_t transpose32(uint32_t x, int lane)
{
    uint32_t o;
    o = lane_xor<16>(x);
    x = (lane & 16) ? ((x & 0xFFFF0000u) | ((o >> 16) & 0x0000FFFFu)) : ((x & 0x0000FFFFu) | ((o & 0x0000FFFFu) << 16));
    o = lane_xor<8>(x);
    x = (lane & 8) ? ((x & 0xFF00FF00u) | ((o >> 8) & 0x00FF00FFu)) : ((x & 0x00FF00FFu) | ((o & 0x00FF00FFu) << 8));
    o = lane_xor<4>(x);
    x = (lane & 4) ? ((x & 0xF0F0F0F0u) | ((o >> 4) & 0x0F0F0F0Fu)) : ((x & 0x0F0F0F0Fu) | ((o & 0x0F0F0F0Fu) << 4));
    o = lane_xor<2>(x);
    x = (lane & 2) ? ((x & 0xCCCCCCCCu) | ((o >> 2) & 0x33333333u)) : ((x & 0x33333333u) | ((o & 0x33333333u) << 2));
    o = lane_xor<1>(x);
    x = (lane & 1) ? ((x & 0xAAAAAAAAu) | ((o >> 1) & 0x55555555u)) : ((x & 0x55555555u) | ((o & 0x55555555u) << 1));
    return x;
}

template <int NG, int LG, bool PB16>
__device__ __forceinline__ void fr_coords(const DevPlan& P, const Wave& W, int tt, int Wn, bool first, int pbpos, int pbn);
template <int NG, int LG, bool PB16, int FRU>
__device__ __forceinline__ void fr_coords1(const DevPlan& P, const Wave& W, int tt, int pbpos, int pbn);

// Table decode ("four Russians") of the n <= fr_cap slots listed in
// W.fri / W.frc for token tt.  For a coordinate iota the signs of the listed
// slots form bit words U(iota), bit j = parity(M_iota & fri[j]) (App. A.4,
// packed-parity equation).  Parity is linear in M_iota, so each word is the
// XOR of one table row per 4-bit group of M_iota; the tables (frv) come from
// the bit transpose of the listed indices.  The decode at iota is then
//     y[iota] = (1/sqrt d) sum_j frc[j] (-1)^U_j(iota),
// summed four slots at a time from 16-entry tables of signed sums (frt).
// `first` overwrites y, otherwise adds.  When pbn > 0, bits pbpos ..
// pbpos + pbn - 1 of U (the leaf level's parents) are stored in W.pb.
// NG = number of 4-bit groups of the widest index.
template <int NG, bool PB16, int FRU>
__device__ void fr_chunk(const DevPlan& P, const Wave& W, int tt, int n, bool first, int pbpos, int pbn)
{
    const int lane = W.lane, dp = P.dp;
    const int Wn = (n + 31) >> 5;
    // slot-parity tables: frv[w][g][v] = bits over the slots of word w of parity(idx & (v << 4g))
    for (int h = 0; 64 * h < n; ++h) {
        const int j = 64 * h + lane;
        const uint32_t x = j < n ? (uint32_t)W.fri[j] : 0u;
        const uint32_t E = transpose32(x, lane);
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
            const int w = 2 * h + hh;
            if (w >= Wn) break;
#pragma unroll
            for (int pass = 0; pass < (NG + 3) / 4; ++pass) {
                const int g = 4 * pass + (lane >> 4), v = lane & 15;
                uint32_t V = 0;
#pragma unroll
                for (int b = 0; b < 4; ++b) {
                    const uint32_t e = (uint32_t)__shfl((int)E, 32 * hh + 4 * g + b, 64);
                    if ((v >> b) & 1) V ^= e;
                }
                if (g < NG) W.frv[(w * 8 + g) * 16 + v] = V;
            }
        }
    }
    // signed sums of four coefficients: frt[i][v] = rsd * sum_b (-1)^(v_b) frc[4i + b],
    // for every group of the used words (groups past n are zero)
    for (int i0 = 0; i0 < 8 * Wn; i0 += 4) {
        const int i = i0 + (lane >> 4), v = lane & 15;
        const float4 c = *(const float4*)(W.frc + 4 * i);
        const float t0 = __uint_as_float(__float_as_uint(c.x) ^ ((uint32_t)(v & 1) << 31)) +
                         __uint_as_float(__float_as_uint(c.y) ^ ((uint32_t)((v >> 1) & 1) << 31));
        const float t1 = __uint_as_float(__float_as_uint(c.z) ^ ((uint32_t)((v >> 2) & 1) << 31)) +
                         __uint_as_float(__float_as_uint(c.w) ^ ((uint32_t)((v >> 3) & 1) << 31));
        W.frt[i * 16 + v] = P.rsd * (t0 + t1);
    }
    wave_sync();

    // a single word with at most 24 slots skips its last two groups
    if (Wn == 1 && first && pbn > 0) {
        if (n <= 24) fr_coords1<NG, 6, PB16, FRU>(P, W, tt, pbpos, pbn);
        else fr_coords1<NG, 8, PB16, FRU>(P, W, tt, pbpos, pbn);
    } else if (Wn == 1 && n <= 24) {
        fr_coords<NG, 6, PB16>(P, W, tt, Wn, first, pbpos, pbn);
    } else {
        fr_coords<NG, 8, PB16>(P, W, tt, Wn, first, pbpos, pbn);
    }
    wave_sync();
}

// Coordinate loop of the table decode over Wn words; LG (even, <= 8) groups
// of each word are summed (the others hold no slot).  Two coordinates at a
// time, all their table reads ahead of their writes.
template <int NG, int LG, bool PB16>
__device__ __forceinline__ void fr_coords(const DevPlan& P, const Wave& W, int tt, int Wn, bool first, int pbpos, int pbn)
{
    const int lane = W.lane, dp = P.dp;
    const uint32_t vbase = lds_addr(W.frv), tbase = lds_addr(W.frt);
    float* yt = W.y + tt * dp;
    const int w0 = pbpos >> 5, sh = pbpos & 31;
    const uint32_t pmask = pbn >= 32 ? ~0u : ((1u << pbn) - 1u);
    auto eval = [&](int iota, float& acc, uint32_t& lo, uint32_t& hi) {
        // 4 x nibble g of the row mask: even groups in s0, odd groups in s1, byte g / 2
        const uint32_t M = W.mask[iota];
        const uint32_t s0 = (M << 2) & 0x3C3C3C3Cu, s1 = (M >> 2) & 0x3C3C3C3Cu;
        acc = 0.f;
        lo = 0;
        hi = 0;
        for (int w = 0; w < Wn; ++w) {
            const uint32_t vb = vbase + (uint32_t)(w * 512), tb = tbase + (uint32_t)(w * 512);
            uint32_t U = 0;
#pragma unroll
            for (int g = 0; g < NG; ++g)
                U ^= lds_ld(__builtin_amdgcn_perm(vb, (g & 1) ? s1 : s0, 0x07060500u | (uint32_t)(g >> 1)) +
                            (uint32_t)(g * 64));
            const uint32_t e4 = (U << 2) & 0x3C3C3C3Cu, o4 = (U >> 2) & 0x3C3C3C3Cu;
#pragma unroll
            for (int i8 = 0; i8 < LG; ++i8)
                acc += lds_ldf(__builtin_amdgcn_perm(tb, (i8 & 1) ? o4 : e4, 0x07060500u | (uint32_t)(i8 >> 1)) + (uint32_t)(i8 * 64));
            lo = w == w0 ? U : lo;
            hi = w == w0 + 1 ? U : hi;
        }
    };
    auto store = [&](int iota, float acc, uint32_t lo, uint32_t hi) {
        if (first) yt[iota] = acc;
        else yt[iota] += acc;
        if (pbn > 0) {
            const uint32_t bits = (sh ? ((lo >> sh) | (hi << (32 - sh))) : lo) & pmask;
            if constexpr (PB16) ((uint16_t*)W.pb)[tt * dp + iota] = (uint16_t)bits;
            else ((uint8_t*)W.pb)[tt * dp + iota] = (uint8_t)bits;
        }
    };
    int iota = lane;
    for (; iota + 64 < dp; iota += 128) {
        float a0, a1;
        uint32_t l0, h0, l1, h1;
        eval(iota, a0, l0, h0);
        eval(iota + 64, a1, l1, h1);
        store(iota, a0, l0, h0);
        store(iota + 64, a1, l1, h1);
    }
    if (iota < dp) {
        float a;
        uint32_t l, h;
        eval(iota, a, l, h);
        store(iota, a, l, h);
    }
}

// The common case of the coordinate loop: one word, the first write of y,
// the leaf parents' sign bits inside the word.  FRU coordinates at a time:
// every table read of the group is issued before any of its writes (the
// compiler cannot reorder reads past stores to the same LDS), so their
// latencies overlap.
template <int NG, int LG, bool PB16, int FRU>
__device__ __forceinline__ void fr_coords1(const DevPlan& P, const Wave& W, int tt, int pbpos, int pbn)
{
    const int lane = W.lane, dp = P.dp;
    const uint32_t vb = lds_addr(W.frv), tb = lds_addr(W.frt);
    float* yt = W.y + tt * dp;
    const uint32_t pmask = (1u << pbn) - 1u;   // pbpos + pbn <= 32
    auto word = [&](int iota) {
        const uint32_t M = W.mask[iota];
        const uint32_t s0 = (M << 2) & 0x3C3C3C3Cu, s1 = (M >> 2) & 0x3C3C3C3Cu;
        uint32_t U = 0;
#pragma unroll
        for (int g = 0; g < NG; ++g)
            U ^= lds_ld(__builtin_amdgcn_perm(vb, (g & 1) ? s1 : s0, 0x07060500u | (uint32_t)(g >> 1)) + (uint32_t)(g * 64));
        return U;
    };
    auto sum = [&](uint32_t U) {
        const uint32_t e4 = (U << 2) & 0x3C3C3C3Cu, o4 = (U >> 2) & 0x3C3C3C3Cu;
        float acc = lds_ldf(__builtin_amdgcn_perm(tb, e4, 0x07060500u));
#pragma unroll
        for (int i8 = 1; i8 < LG; ++i8)
            acc += lds_ldf(__builtin_amdgcn_perm(tb, (i8 & 1) ? o4 : e4, 0x07060500u | (uint32_t)(i8 >> 1)) + (uint32_t)(i8 * 64));
        return acc;
    };
    auto store = [&](int iota, uint32_t U, float acc) {
        yt[iota] = acc;
        const uint32_t bits = (U >> pbpos) & pmask;
        if constexpr (PB16) ((uint16_t*)W.pb)[tt * dp + iota] = (uint16_t)bits;
        else ((uint8_t*)W.pb)[tt * dp + iota] = (uint8_t)bits;
    };
    int iota = lane;
    for (; iota + 64 * (FRU - 1) < dp; iota += 64 * FRU) {
        uint32_t U[FRU];
        float acc[FRU];
#pragma unroll
        for (int u = 0; u < FRU; ++u) U[u] = word(iota + 64 * u);
#pragma unroll
        for (int u = 0; u < FRU; ++u) acc[u] = sum(U[u]);
#pragma unroll
        for (int u = 0; u < FRU; ++u) store(iota + 64 * u, U[u], acc[u]);
    }
    for (; iota < dp; iota += 64) {
        const uint32_t U = word(iota);
        store(iota, U, sum(U));
    }
}

// Gamma^T alpha of the last level's columns on the matrix cores (16x16x16,
// alpha split exactly into bf16 terms), each column multiplied by its
// parent's signs (bits of W.pb) and added to y.  A lane holds four columns
// of one token at one coordinate; the lanes of a token's CPT columns are
// summed by a swizzle (and a permute), after which they hold bit-identical
// sums (each addition is commutative).
template <bool EXACT3>
__device__ __forceinline__ f32x4 column_acc(bf16x4 ahi, bf16x4 amid, bf16x4 alo, u32x2 bfe)
{
    const bf16x4 b = __builtin_bit_cast(bf16x4, bfe);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ahi, b, acc, 0, 0, 0);
    if constexpr (EXACT3) acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(amid, b, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(alo, b, acc, 0, 0, 0);
    return acc;
}

__device__ __forceinline__ float column_signs(f32x4 acc, uint32_t pv)
{
    return (__uint_as_float(__float_as_uint(acc[0]) ^ (pv << 31)) +
            __uint_as_float(__float_as_uint(acc[1]) ^ ((pv >> 1) << 31))) +
           (__uint_as_float(__float_as_uint(acc[2]) ^ ((pv >> 2) << 31)) +
            __uint_as_float(__float_as_uint(acc[3]) ^ ((pv >> 3) << 31)));
}

template <bool EXACT3>
__device__ __forceinline__ float column_sum(bf16x4 ahi, bf16x4 amid, bf16x4 alo, u32x2 bfe, uint32_t pv)
{
    return column_signs(column_acc<EXACT3>(ahi, amid, alo, bfe), pv);
}

// Leaf columns when every lane's column belongs to a live token (CPT
// parents, 16 / CPT tokens, all present): each lane of a token's group
// writes the same sum, so there are no masked stores or branches and the
// compiler overlaps the NB columns of a batch.
template <int CPT, bool EXACT3, bool PB16, int NB>
__device__ __forceinline__ void leaf_columns(const DevPlan& P, const Wave& W, bf16x4 ahi, bf16x4 amid, bf16x4 alo)
{
    constexpr int CSH = CPT == 4 ? 2 : CPT == 8 ? 3 : 4;
    const int L1 = P.levels - 1, dp = P.dp, lane = W.lane;
    const int row = lane & 15, grp = lane >> 4;
    const u32x2* bfr = (const u32x2*)P.gamma_t + P.gamma_t_off[L1] + lane;
    const int tok = (4 * grp) >> CSH, q0 = (4 * grp) & (CPT - 1);
    const int pbo = tok * dp + row;
    float* yt = W.y + pbo;
    const int x32 = ((lane ^ 32) << 2);
    const int ncb = dp / 16;
    auto pb_at = [&](int cb) -> uint32_t {
        if constexpr (PB16) return (uint32_t)((const uint16_t*)W.pb)[pbo + 16 * cb] >> q0;
        else return (uint32_t)((const uint8_t*)W.pb)[pbo + 16 * cb] >> q0;
    };
    auto token_sum = [&](float v) {
        if constexpr (CPT >= 8) v += swz_xorf16(v);
        if constexpr (CPT >= 16) v += __int_as_float(__builtin_amdgcn_ds_bpermute(x32, __float_as_int(v)));
        return v;
    };
    int cb0 = 0;
    for (; cb0 + NB <= ncb; cb0 += NB) {
        u32x2 bf[NB];
        uint32_t pbv[NB];
#pragma unroll
        for (int e = 0; e < NB; ++e) {
            bf[e] = bfr[(int64_t)(cb0 + e) * 64];
            pbv[e] = pb_at(cb0 + e);
        }
        // four columns' products in flight at once, in accumulators of their own
        float v[NB];
#pragma unroll
        for (int e0 = 0; e0 < NB; e0 += 4) {
            f32x4 acc[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) acc[u] = column_acc<EXACT3>(ahi, amid, alo, bf[e0 + u]);
#pragma unroll
            for (int u = 0; u < 4; ++u) v[e0 + u] = token_sum(column_signs(acc[u], pbv[e0 + u]));
        }
#pragma unroll
        for (int e = 0; e < NB; ++e) yt[16 * (cb0 + e)] += P.rsd * v[e];
    }
    for (int cb = cb0; cb < ncb; ++cb)   // the last, partial batch
        yt[16 * cb] += P.rsd * token_sum(column_sum<EXACT3>(ahi, amid, alo, bfr[(int64_t)cb * 64], pb_at(cb)));
}

// Leaf columns in general: CPT from the plan, one writer lane per token and
// coordinate, none for absent tokens.
template <bool EXACT3, bool PB16>
__device__ __forceinline__ void leaf_columns_any(const DevPlan& P, const Wave& W, bf16x4 ahi, bf16x4 amid, bf16x4 alo)
{
    const int L1 = P.levels - 1, TPW = P.wave_tokens, dp = P.dp, lane = W.lane;
    const int row = lane & 15, grp = lane >> 4;
    const int CPT = P.cpt[L1];
    const u32x2* bfr = (const u32x2*)P.gamma_t + P.gamma_t_off[L1] + lane;
    const int tok = (4 * grp) >> P.cpt_shift[L1], q0 = (4 * grp) & (CPT - 1);
    const bool writer = (grp & ((CPT >> 2) - 1)) == 0 && tok < W.ntok;
    const int pbo = (tok < TPW ? tok : 0) * dp + row;
    float* yt = W.y + pbo;
    const int x32 = ((lane ^ 32) << 2);
    const int ncb = dp / 16;
    for (int cb0 = 0; cb0 < ncb; cb0 += kBatch) {
        u32x2 bf[kBatch];
        uint32_t pbv[kBatch];
#pragma unroll
        for (int e = 0; e < kBatch; ++e) {
            const int cb = cb0 + e < ncb ? cb0 + e : ncb - 1;
            bf[e] = bfr[(int64_t)cb * 64];
            if constexpr (PB16) pbv[e] = (uint32_t)((const uint16_t*)W.pb)[pbo + 16 * cb] >> q0;
            else pbv[e] = (uint32_t)((const uint8_t*)W.pb)[pbo + 16 * cb] >> q0;
        }
#pragma unroll
        for (int e = 0; e < kBatch; ++e) {
            float v = column_sum<EXACT3>(ahi, amid, alo, bf[e], pbv[e]);
            if (CPT >= 8) v += swz_xorf16(v);
            if (CPT >= 16) v += __int_as_float(__builtin_amdgcn_ds_bpermute(x32, __float_as_int(v)));
            if (writer && cb0 + e < ncb) yt[16 * (cb0 + e)] += P.rsd * v;
        }
    }
}

// Decode of the wave's tokens from W.idx and coefficients `cf` into W.y.
// W.route holds the routes of the last level's slots (when decoding through
// leaf columns).  PB16: the leaf parents' sign bits take 16 bits (else 8).
template <bool EXACT3, int NG, bool PB16, int LCB, int FRU>
__device__ void decode_tokens(const DevPlan& P, const Wave& W, const float* cf)
{
    const int k = P.k_tot, d = P.d, dp = P.dp, TPW = P.wave_tokens, lane = W.lane;
    const int L1 = P.levels - 1;
    const bool cols = P.leaf_columns != 0;
    const int sbL = cols ? P.slot_base[L1] : k;
    const int row = lane & 15, grp = lane >> 4;

    // leaf columns: claim (row, j) cells, then take the column coefficients into
    // matrix-core A fragments (alpha and claims live in the y region until then)
    bf16x4 ahi = {}, amid = {}, alo = {};
    if (cols) {
        const int Kc = P.active[L1 - 1], CPT = P.cpt[L1], KL = P.active[L1];
        const int sbP = P.slot_base[L1 - 1];
        if (lane < 16) {
            const int tt = lane >> P.cpt_shift[L1], q = lane & (CPT - 1);
            W.par[lane] = (tt < W.ntok && q < Kc) ? W.idx[tt * k + sbP + q] : -1;
        }
        for (int i = lane; i < 16 * 16; i += 64) {
            W.alpha[i] = 0.f;
            W.claim[i] = 0x7FFFFFFF;
        }
        wave_sync();
        for (int tt = 0; tt < W.ntok; ++tt)
            for (int s = sbL + lane; s < sbL + KL; s += 64) {
                const int rt = W.route[tt * k + s];
                if (rt >= 0) atomicMin(&W.claim[(tt * CPT + (rt >> 16)) * 16 + (rt & 0xFFFF)], s);
            }
        wave_sync();
        for (int tt = 0; tt < W.ntok; ++tt)
            for (int s = sbL + lane; s < sbL + KL; s += 64) {
                const int rt = W.route[tt * k + s];
                const int at = rt >= 0 ? (tt * CPT + (rt >> 16)) * 16 + (rt & 0xFFFF) : 0;
                const bool mine = rt >= 0 && W.claim[at] == s;
                if (mine) {
                    W.alpha[at] = cf[tt * k + s];
                    W.route[tt * k + s] = rt | kClaimed;
                }
            }
        wave_sync();
        uint32_t h[4] = {0, 0, 0, 0}, m[4] = {0, 0, 0, 0}, lo[4] = {0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float a = W.alpha[row * 16 + 4 * grp + i];
            if constexpr (EXACT3) {
                split3(a, h[i], m[i], lo[i]);
            } else {
                h[i] = f32_to_bf16_rne(a);
                lo[i] = f32_to_bf16_rne(a - bf16_bits_to_f32(h[i]));
            }
        }
        ahi = __builtin_bit_cast(bf16x4, (u32x2){h[0] | (h[1] << 16), h[2] | (h[3] << 16)});
        amid = __builtin_bit_cast(bf16x4, (u32x2){m[0] | (m[1] << 16), m[2] | (m[3] << 16)});
        alo = __builtin_bit_cast(bf16x4, (u32x2){lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16)});
        wave_sync();
    }

    // table decode of every non-basis slot not taken by a column, in chunks of
    // fr_cap.  The leaf parents (slots sbP .. sbL - 1) are always listed, at
    // consecutive positions from pbpos, for their sign bits.
    const int sbP = cols ? P.slot_base[L1 - 1] : k, pbn = cols ? P.active[L1 - 1] : 0, cap = P.fr_cap;
    for (int tt = 0; tt < W.ntok; ++tt) {
        const int32_t* it = W.idx + tt * k;
        const int32_t* rt = W.route + tt * k;
        const float* ct = cf + tt * k;
        int pbpos = 0;
        for (int cs = 0;; cs += cap) {
            int base = 0;
            for (int s0 = 0; s0 < k; s0 += 64) {
                const int s = s0 + lane;
                const int32_t c = s < k ? it[s] : -1;
                const bool claimed = s < k && rt[s] >= 0 && (rt[s] & kClaimed);
                const bool take = s < k && ((s >= sbP && s < sbL) || (c >= d && (s < sbL || !claimed)));
                const uint64_t m = __ballot(take);
                if (s0 <= sbP && sbP < s0 + 64) pbpos = base + (int)__popcll(m & ((1ull << (sbP - s0)) - 1ull));
                const int pos = base + (int)__popcll(m & ((1ull << lane) - 1ull)) - cs;
                if (take && pos >= 0 && pos < cap) {
                    W.fri[pos] = c > 0 ? c : 0;
                    W.frc[pos] = c >= d ? ct[s] : 0.f;
                }
                base += (int)__popcll(m);
            }
            const int n = max(0, min(base - cs, cap));
            for (int j = n + lane; j < ((n + 31) & ~31); j += 64) W.frc[j] = 0.f;  // zero the rest of the last word
            wave_sync();
            fr_chunk<NG, PB16, FRU>(P, W, tt, n, cs == 0, pbpos - cs, (pbpos >= cs && pbpos < cs + cap) ? pbn : 0);
            if (base <= cs + cap) break;
        }
    }

    if (cols) {
        // Gamma^T alpha on the matrix cores, then the parents' signs.  With
        // every column a live token's (full waves of two tokens of eight
        // parents) all lanes write.
        const int CPT = P.cpt[L1];
        const bool all = TPW * CPT == 16 && W.ntok == TPW;
        // (one compile-time layout per kernel variant: more of them inlined here
        // cost the kernels registers, and with them a wave per SIMD.  Eight
        // parents per token take one byte of sign bits (PB16 false), sixteen
        // take two: one token per wave, all sixteen columns its own)
        if (!PB16 && CPT == 8 && all) leaf_columns<8, EXACT3, PB16, LCB>(P, W, ahi, amid, alo);
        else if (PB16 && CPT == 16 && all) leaf_columns<16, EXACT3, PB16, LCB>(P, W, ahi, amid, alo);
        else leaf_columns_any<EXACT3, PB16>(P, W, ahi, amid, alo);
        wave_sync();
    }

    // basis slots: coefficient at their own coordinate.  Distinct
    // coordinates (the encoder's level 0) are added by all lanes at once; a
    // block with a repeated coordinate adds its slots one by one, in slot order.
    for (int tt = 0; tt < W.ntok; ++tt)
        for (int s0 = 0; s0 < k; s0 += 64) {
            const int s = s0 + lane;
            const int32_t c = s < k ? W.idx[tt * k + s] : -1;
            const int a = s < k ? __float_as_int(cf[tt * k + s]) : 0;
            const bool basis = c >= 0 && c < d;
            uint64_t m = __ballot(basis);
            if (!m) continue;
            bool dup = false;
            if (cols) {
                // the leaf parents' sign bytes are dead now: each basis lane
                // marks its coordinate; a lane that reads back another lane's
                // mark shares the coordinate with it
                uint8_t* mark = (uint8_t*)W.pb + tt * dp;
                if (basis) mark[c] = (uint8_t)lane;
                wave_sync();
                dup = basis && mark[c] != (uint8_t)lane;
            } else {
                for (uint64_t mm = m; mm; mm &= mm - 1) {
                    const int b = __builtin_ctzll(mm);
                    dup |= basis && b < lane && rdlane(c, b) == c;
                }
            }
            if (!__ballot(dup)) {
                if (basis) W.y[tt * dp + c] += __int_as_float(a);
            } else {
                while (m) {
                    const int b = __builtin_ctzll(m);
                    m &= m - 1;
                    const int cb = rdlane(c, b);
                    const float ab = __int_as_float(rdlane(a, b));
                    if (lane == 0) W.y[tt * dp + cb] += ab;
                }
            }
            wave_sync();
        }
    wave_sync();
}

__device__ Wave make_wave(const DevPlan& P, unsigned char* smem, bool scoring, bool act_bf16, int wave, int lane)
{
    const CodeLayout CL = code_layout(P, scoring, act_bf16);
    unsigned char* b = smem + code_shared_bytes(P) + (unsigned)wave * CL.bytes;
    Wave W;
    W.lane = lane;
    W.t0 = 0;
    W.ntok = 0;
    W.idx = (int32_t*)(b + CL.idx);
    W.coef = (float*)(b + CL.coef);
    W.route = (int32_t*)(b + CL.route);
    W.par = (int32_t*)(b + CL.par);
    W.alpha = (float*)(b + CL.alpha);
    W.claim = (int32_t*)(b + CL.claim);
    W.fri = (int32_t*)(b + CL.fri);
    W.frc = (float*)(b + CL.frc);
    W.frv = (uint32_t*)(b + CL.frv);
    W.frt = (float*)(b + CL.frt);
    W.pb = (void*)(b + CL.pb);
    W.y = (float*)(b + CL.y);
    W.pairs = (uint32_t*)(b + CL.pairs);
    W.gf = (float*)(b + CL.y);
    W.cw = (uint32_t*)(b + CL.cw);
    W.score = (float*)(b + CL.score);
    const unsigned o_gtab = align16u(P.dp * 4);
    const unsigned o_gens = o_gtab + align16u(P.gtab_total * 8);
    W.mask = (const uint32_t*)smem;
    W.gtab = (const uint32_t*)(smem + o_gtab);
    W.gens = (const uint32_t*)(smem + o_gens);
    return W;
}

// a, b += the 8 elements of `add` at i (fewer when rem < 8, vec false).
template <bool BF16>
__device__ __forceinline__ void add_row8(const void* add, int64_t i, int rem, bool vec, float4& a, float4& b)
{
    float v[8];
    if (vec) {
        if constexpr (BF16) {
            const u32x4 q = *(const u32x4*)((const uint16_t*)add + i);
            const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[2 * e] = bf16_bits_to_f32(w[e] & 0xFFFFu);
                v[2 * e + 1] = bf16_bits_to_f32(w[e] >> 16);
            }
        } else {
            const float4 p = *(const float4*)((const float*)add + i), q = *(const float4*)((const float*)add + i + 4);
            v[0] = p.x; v[1] = p.y; v[2] = p.z; v[3] = p.w;
            v[4] = q.x; v[5] = q.y; v[6] = q.z; v[7] = q.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = e < rem ? load_act<BF16>(add, i + e) : 0.f;
    }
    a.x += v[0]; a.y += v[1]; a.z += v[2]; a.w += v[3];
    b.x += v[4]; b.y += v[5]; b.z += v[6]; b.w += v[7];
}

// Converts the wave's fp32 rows to the output type, 8 coordinates per lane
// (16- or 32-byte stores when d is a multiple of 8).  A non-null `add`
// (same type and shape as out) is added first; it may alias out.
template <bool OUT_BF16>
__device__ void write_rows(const DevPlan& P, const Wave& W, void* out, const void* add = nullptr)
{
    const int d = P.d, dp = P.dp;
    const bool vec = (d & 7) == 0;
    for (int tt = 0; tt < W.ntok; ++tt) {
        const float* yt = W.y + tt * dp;
        const int64_t r0 = (W.t0 + tt) * d;
        for (int o = W.lane * 8; o < d; o += 512) {
            float4 a = *(const float4*)(yt + o), b = *(const float4*)(yt + o + 4);
            if (add) add_row8<OUT_BF16>(add, r0 + o, d - o, vec, a, b);
            if (vec) {
                if constexpr (OUT_BF16) {
                    u32x4 v;
                    v.x = pack_bf16x2(a.x, a.y);
                    v.y = pack_bf16x2(a.z, a.w);
                    v.z = pack_bf16x2(b.x, b.y);
                    v.w = pack_bf16x2(b.z, b.w);
                    *(u32x4*)((uint16_t*)out + r0 + o) = v;
                } else {
                    *(float4*)((float*)out + r0 + o) = a;
                    *(float4*)((float*)out + r0 + o + 4) = b;
                }
            } else {
                const float v[8] = {a.x, a.y, a.z, a.w, b.x, b.y, b.z, b.w};
#pragma unroll
                for (int e = 0; e < 8; ++e)
                    if (o + e < d) store_act<OUT_BF16>(out, r0 + o + e, v[e]);
            }
        }
    }
}

__device__ void load_shared(const DevPlan& P, unsigned char* smem)
{
    const unsigned o_gtab = align16u(P.dp * 4);
    const unsigned o_gens = o_gtab + align16u(P.gtab_total * 8);
    uint32_t* s_mask = (uint32_t*)smem;
    uint32_t* s_gtab = (uint32_t*)(smem + o_gtab);
    uint32_t* s_gens = (uint32_t*)(smem + o_gens);
    for (int i = threadIdx.x; i < P.dp; i += kThreads) s_mask[i] = P.masks[i];
    for (int i = threadIdx.x; i < 2 * P.gtab_total; i += kThreads) s_gtab[i] = P.gtab[i];
    for (int i = threadIdx.x; i < P.gens_total; i += kThreads) s_gens[i] = P.gens[i];
    __syncthreads();
}

// Loads the codes of the wave's tokens into LDS and resets routes.
__device__ void load_codes(const DevPlan& P, const Wave& W, const int32_t* idx, const float* coef)
{
    const int k = P.k_tot, TPW = P.wave_tokens;
    for (int tt = 0; tt < TPW; ++tt) {
        const bool live = tt < W.ntok;
        for (int s = W.lane; s < k; s += 64) {
            W.idx[tt * k + s] = live ? idx[(W.t0 + tt) * k + s] : -1;
            if (coef) W.coef[tt * k + s] = live ? coef[(W.t0 + tt) * k + s] : 0.f;
            W.route[tt * k + s] = -1;
        }
    }
}

template <bool OUT_BF16, int NG, bool PB16>
__global__ __launch_bounds__(kThreads) void decode2_kernel(DevPlan P, const int32_t* __restrict__ idx,
                                                           const float* __restrict__ coef, int64_t T,
                                                           void* __restrict__ y)
{
    extern __shared__ __align__(16) unsigned char smem[];
    load_shared(P, smem);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, TPW = P.wave_tokens, k = P.k_tot;
    Wave W = make_wave(P, smem, false, true, wave, lane);
    const int64_t ngroups = (T + TPW - 1) / TPW;
    const int64_t gstride = (int64_t)gridDim.x * kCodeWaves;
    // the next group's code is requested while this group is decoded (two
    // tokens of at most 128 slots or one of at most 256: four words of each
    // array per lane)
    constexpr int kPrefetch = 4;
    const bool pf = (TPW == 2 && k <= 128) || (TPW == 1 && k <= 256);
    int32_t nidx[kPrefetch];
    float ncoef[kPrefetch];
    auto fetch = [&](int64_t grp) {
#pragma unroll
        for (int e = 0; e < kPrefetch; ++e) {
            const int tt = TPW == 2 ? e >> 1 : 0, s = (TPW == 2 ? (e & 1) : e) * 64 + lane;
            const int64_t t = grp * TPW + tt;
            const bool ok = s < k && t < T;
            nidx[e] = ok ? idx[t * k + s] : -1;
            ncoef[e] = ok ? coef[t * k + s] : 0.f;
        }
    };
    int64_t grp = (int64_t)blockIdx.x * kCodeWaves + wave;
    if (pf && grp < ngroups) fetch(grp);
    for (; grp < ngroups; grp += gstride) {
        W.t0 = grp * TPW;
        W.ntok = (int)min((int64_t)TPW, T - W.t0);
        if (pf) {
#pragma unroll
            for (int e = 0; e < kPrefetch; ++e) {
                const int tt = TPW == 2 ? e >> 1 : 0, s = (TPW == 2 ? (e & 1) : e) * 64 + lane;
                if (s < k) {
                    W.idx[tt * k + s] = nidx[e];
                    W.coef[tt * k + s] = ncoef[e];
                    W.route[tt * k + s] = -1;
                }
            }
            if (grp + gstride < ngroups) fetch(grp + gstride);
        } else {
            load_codes(P, W, idx, coef);
        }
        wave_sync();
        if (P.leaf_columns) {
            route_slots(P, W);
            wave_sync();
        }
        decode_tokens<!OUT_BF16, NG, PB16, kBatch, kDecodeUnroll>(P, W, W.coef);
        write_rows<OUT_BF16>(P, W, y);
        wave_sync();
    }
}

// g at coordinate iota of token tt, from the LDS copy.
template <bool G_BF16>
__device__ __forceinline__ float g_at(const DevPlan& P, const Wave& W, int tt, int iota)
{
    if constexpr (G_BF16) return pair_value(P, W.pairs, tt, iota);
    else return W.gf[tt * P.dp + iota];
}

// Child scores of the parent columns of level l against the wave's g,
// written to the coefficients of the slots routed to them.
template <bool G_BF16>
__device__ void score_level(const DevPlan& P, const Wave& W, int l)
{
    const int k = P.k_tot, TPW = P.wave_tokens, lane = W.lane;
    const int CPT = P.cpt[l], csh = P.cpt_shift[l], Kp = P.active[l - 1], Kl = P.active[l];
    const int ncol = TPW * CPT, NB = (ncol + 15) >> 4, sbp = P.slot_base[l - 1], sbl = P.slot_base[l];
    const ActTile A{W.pairs, W.gf};
    const int col = lane & 15, kq = lane >> 4;
    for (int nb = 0; nb < NB; ++nb) {
        column_bitmaps(P, lane, W.ntok, csh, nb, W.idx + sbp, k, Kp, P.nt, W.cw);
        wave_sync();
        const int r = nb * 16 + col, tt = r >> csh, q = r & (CPT - 1);
        const bool valid = r < ncol && tt < W.ntok && q < Kp && W.idx[tt * k + sbp + q] >= 0;
        const int trow = valid ? tt : 0;
        for (int mb = 0; mb < P.mblocks[l]; ++mb) {
            const f32x4 acc = mfma_scores<G_BF16>(P, lane, l, mb, trow, A, W.cw);
#pragma unroll
            for (int i = 0; i < 4; ++i) W.score[col * 16 + kq * 4 + i] = acc[i] * P.rsd;
            wave_sync();
            // slots routed to a column of this block and a generator of this tile
            for (int tt2 = 0; tt2 < W.ntok; ++tt2)
                for (int s = sbl + lane; s < sbl + Kl; s += 64) {
                    const int rt = W.route[tt2 * k + s];
                    if (rt < 0) continue;
                    const int r2 = (tt2 << csh) + (rt >> 16), j = rt & 0xFFFF;
                    if ((r2 >> 4) == nb && (j >> 4) == mb) W.coef[tt2 * k + s] = W.score[(r2 & 15) * 16 + (j & 15)];
                }
            wave_sync();
        }
    }
}

typedef __bf16 bf16x2v __attribute__((ext_vector_type(2)));

// c + a.lo b.lo + a.hi b.hi for bf16 pairs.  The operands are taken as plain
// words: a bit cast of a vector element (pq.y) reads element 0 with this
// compiler.
__device__ __forceinline__ float dot2u(uint32_t a, uint32_t b, float c)
{
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2v, a), __builtin_bit_cast(bf16x2v, b), c, false);
}

// +-1 bf16 pair carrying bits 15 and 31 of R as its signs
__device__ __forceinline__ uint32_t unit_pair(uint32_t R)
{
    return __builtin_amdgcn_bitop3_b32(R, 0x80008000u, 0x3F803F80u, 0xEA);   // (R & signs) | one
}

// grad_coef of the hashed slots that route nowhere: the scaled sum over the
// coordinates of g(iota) (-1)^{parity(M_iota & c)} for slot index c, with
// one lane per slot while 64 or more remain, then 2, 4 or 8 lanes per slot
// (each taking every 2nd, 4th or 8th chunk) in rounds of 32, 16 and 8 slots,
// so that the lanes stay busy (48 slots: 32 at two lanes, then 16 at four,
// 18 chunk steps instead of 24).  The slot's signs over the 32
// coordinates of chunk w form one word, the XOR of one nibble-table word per
// 4-bit group of c (parity is linear in the index bits).  bf16 g: dword o of
// the chunk holds coordinates o and o + 16, which meet the +-1 pair made from
// word bits o and o + 16 in a two-element dot product (fp32 accumulation).
template <bool G_BF16, int NG>
__device__ void direct_scores(const DevPlan& P, const Wave& W)
{
    static_assert(NG <= kNtGroupsPadded, "nibble groups beyond the padded tables");
    const int k = P.k_tot, n = W.ntok * k, lane = W.lane, nchunk = P.nchunk, d = P.d;
    int32_t* list = (int32_t*)W.score;   // 256 entries
    const uint64_t below = (1ull << lane) - 1;
    for (int w0 = 0; w0 < n; w0 += 256) {
        int m = 0;
        for (int b = w0; b < min(n, w0 + 256); b += 64) {
            const int i = b + lane;
            const bool act = i < n && W.idx[i] >= d && W.route[i] < 0;
            const uint64_t bal = __ballot(act);
            if (act) list[m + __popcll(bal & below)] = i;
            m += __popcll(bal);
        }
        wave_sync();
        for (int r0 = 0; r0 < m;) {
            const int rem = m - r0;
            const int sh = rem >= 64 ? 0 : rem >= 32 ? 1 : rem >= 16 ? 2 : 3;   // 2^sh lanes per slot
            const int mr = min(64 >> sh, rem);
            const int r = lane & ((64 >> sh) - 1), part = lane >> (6 - sh);
            const bool valid = r < mr;
            const int item = list[r0 + (valid ? r : 0)];
            const int tt = item / k;
            const uint32_t c = (uint32_t)W.idx[item];
            float acc0 = 0.f, acc1 = 0.f;
            // the nibble-table words of the next chunk are requested before
            // this chunk is summed (the device tables hold at least NG groups,
            // zero words past nt_groups)
            uint32_t toff[NG], tw[NG];
#pragma unroll
            for (int g = 0; g < NG; ++g) toff[g] = 4u * ((uint32_t)(g * nchunk * 16) + ((c >> (4 * g)) & 15u));
            const unsigned char* ntb = (const unsigned char*)P.nt;   // byte offsets: 32-bit address arithmetic
            auto fetch_words = [&](int w) {
#pragma unroll
                for (int g = 0; g < NG; ++g) tw[g] = *(const uint32_t*)(ntb + (toff[g] + (uint32_t)(w * 64)));
            };
            auto fold_words = [&]() {
                uint32_t v = 0;
#pragma unroll
                for (int g = 0; g < NG; ++g) v ^= tw[g];
                return v;
            };
            fetch_words(min(part, nchunk - 1));
            for (int w = part; w < nchunk; w += 1 << sh) {
                const uint32_t word = fold_words();
                fetch_words(min(w + (1 << sh), nchunk - 1));
                // keeps the compiler from sinking those loads to their use
                __asm__ volatile("" ::: "memory");
                if constexpr (G_BF16) {
                    const u32x4* pr = (const u32x4*)(W.pairs + tt * P.prow + w * 16);
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const u32x4 pq = pr[q];
                        const int o = 4 * q;
                        acc0 = dot2u(pq.x, unit_pair(word << (15 - o)), acc0);
                        acc1 = dot2u(pq.y, unit_pair(word << (14 - o)), acc1);
                        acc0 = dot2u(pq.z, unit_pair(word << (13 - o)), acc0);
                        acc1 = dot2u(pq.w, unit_pair(word << (12 - o)), acc1);
                    }
                } else {
                    const float* gr = W.gf + tt * P.dp + 32 * w;
#pragma unroll
                    for (int b = 0; b < 32; b += 2) {
                        acc0 += __uint_as_float(__float_as_uint(gr[b]) ^ ((word << (31 - b)) & 0x80000000u));
                        acc1 += __uint_as_float(__float_as_uint(gr[b + 1]) ^ ((word << (30 - b)) & 0x80000000u));
                    }
                }
            }
            float acc = acc0 + acc1;
            for (int off = 64 >> sh; off < 64; off <<= 1) acc += __shfl_xor(acc, off, 64);
            if (valid && part == 0) W.coef[item] = P.rsd * acc;
            r0 += mr;
        }
        wave_sync();   // the list is rewritten by the next window
    }
}

// PF1: the next group's code is prefetched for waves of one token (a
// separate instance: selecting the layout at run time costs the two-token
// form a wave per SIMD in registers).
template <bool G_BF16, bool GX_BF16, int NG, bool PB16, bool PF1 = false>
__global__ __launch_bounds__(kThreads) void decode_bwd2_kernel(DevPlan P, const int32_t* __restrict__ idx,
                                                               const void* __restrict__ g, int64_t T,
                                                               float* __restrict__ grad_coef,
                                                               void* grad_x, const float* __restrict__ add_gc,
                                                               const void* add_gx,
                                                               const float2* __restrict__ stats)
{
    extern __shared__ __align__(16) unsigned char smem[];
    load_shared(P, smem);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, TPW = P.wave_tokens, k = P.k_tot;
    const int d = P.d, dp = P.dp;
    Wave W = make_wave(P, smem, true, G_BF16, wave, lane);
    const int64_t ngroups = (T + TPW - 1) / TPW;
    const int64_t gstride = (int64_t)gridDim.x * kCodeWaves;
    // the next group's code is requested while this group is processed
    // (two tokens of at most 128 slots, or with PF1 one of at most 256: four
    // words per lane)
    const bool pf = PF1 ? (TPW == 1 && k <= 256) : (TPW == 2 && k <= 128);
    int32_t nidx[4];
    auto fetch = [&](int64_t gp) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int tt = PF1 ? 0 : e >> 1, s = (PF1 ? e : (e & 1)) * 64 + lane;
            const int64_t t = gp * TPW + tt;
            nidx[e] = (s < k && t < T) ? idx[t * k + s] : -1;
        }
    };
    int64_t grp = (int64_t)blockIdx.x * kCodeWaves + wave;
    if (pf && grp < ngroups) fetch(grp);
    for (; grp < ngroups; grp += gstride) {
        const int64_t t0 = grp * TPW;
        W.t0 = t0;
        W.ntok = (int)min((int64_t)TPW, T - t0);

        // codes, routes reset, and g in LDS
        if (pf) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int tt = PF1 ? 0 : e >> 1, s = (PF1 ? e : (e & 1)) * 64 + lane;
                if (s < k) {
                    W.idx[tt * k + s] = nidx[e];
                    W.route[tt * k + s] = -1;
                }
            }
            if (grp + gstride < ngroups) fetch(grp + gstride);
        } else {
            load_codes(P, W, idx, nullptr);
        }
        if constexpr (G_BF16) {
            load_pairs(P, lane, W.ntok, TPW, (const uint16_t*)g, t0, W.pairs);
        } else {
            const float* gfp = (const float*)g;
            for (int tt = 0; tt < TPW; ++tt)
                for (int iota = lane; iota < dp; iota += 64)
                    W.gf[tt * dp + iota] = (tt < W.ntok && iota < d) ? gfp[(t0 + tt) * d + iota] : 0.f;
        }
        wave_sync();

        // route the last level's slots to a parent slot of the previous level
        // (its scoring and the decode's leaf columns use the routes; plans with
        // many children per parent take every slot directly below)
        if (!P.bwd_direct) route_slots(P, W);
        // coefficients for basis slots and padding
        for (int tt = 0; tt < TPW; ++tt)
            for (int s = lane; s < k; s += 64) {
                const int32_t c = W.idx[tt * k + s];
                float v = 0.f;
                if (tt < W.ntok && c >= 0 && c < d) v = g_at<G_BF16>(P, W, tt, c);
                W.coef[tt * k + s] = v;
            }
        wave_sync();

        // grad_coef of routed slots: child scores of each parent column against g
        if (!P.bwd_direct && P.levels > 1) score_level<G_BF16>(P, W, P.levels - 1);

        // hashed slots that are not routed (levels below the last, slots that
        // route nowhere, every hashed slot when the plan has many children per
        // parent): direct reductions over the coordinates
        direct_scores<G_BF16, NG>(P, W);
        wave_sync();
        if (add_gc) {
            for (int i = lane; i < W.ntok * k; i += 64) W.coef[i] += add_gc[t0 * k + i];
            wave_sync();
        }
        for (int i = lane; i < W.ntok * k; i += 64) grad_coef[t0 * k + i] = W.coef[i];
        if (stats) {
            // standardized coefficients z = (s - mu) r: dz/dx = r phi
            wave_sync();
            const int32_t nfeat_sh = P.level_bits[P.levels - 1];
            for (int i = lane; i < W.ntok * k; i += 64) {
                const int32_t c = W.idx[i];
                if (c >= 0 && (c >> nfeat_sh) == 0) W.coef[i] *= stats[c].y;
            }
            wave_sync();
        }

        // grad_x = decode(idx, grad_coef) (+ add_gx); the scoring buffers are dead now
        decode_tokens<!GX_BF16, NG, PB16, kBwdBatch, kDecodeUnroll>(P, W, W.coef);
        write_rows<GX_BF16>(P, W, grad_x, add_gx);
        wave_sync();
    }
}

size_t code_lds_bytes(const DevPlan& P, bool scoring, bool act_bf16)
{
    return code_shared_bytes(P) + (size_t)kCodeWaves * code_layout(P, scoring, act_bf16).bytes;
}

int device_cus()
{
    static int cus = 0;
    if (!cus) {
        int dev = 0;
        hipDeviceProp_t prop;
        if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
            cus = prop.multiProcessorCount;
        if (cus <= 0) cus = 256;
    }
    return cus;
}

// Grid-stride launch: `rounds` times the workgroups the chip holds at once
// (measured best: one round for the decode, four for the backward).
dim3 code_grid(const DevPlan& P, int64_t T, size_t lds, int rounds)
{
    const int64_t groups = (T + P.wave_tokens - 1) / P.wave_tokens;
    const int64_t need = (groups + kCodeWaves - 1) / kCodeWaves;
    const int per_cu = lds ? (int)std::max<size_t>(1, (160 * 1024) / lds) : 4;
    const int64_t cap = (int64_t)device_cus() * std::min(per_cu, 8) * rounds;
    return dim3((unsigned)std::max<int64_t>(1, std::min(need, cap)));
}

}  // namespace

static bool code_rows_fit(const DevPlan& P)
{
    return code_lds_bytes(P, true, true) <= (size_t)kLdsBudget && code_lds_bytes(P, true, false) <= (size_t)kLdsBudget;
}

// The plan as the code kernels take it: a wave keeps the encoder's
// wave_tokens tokens (16 parent columns) where their rows fit the LDS budget;
// wide rows with few parents per token (d in the thousands, K_0 of 2 or 4)
// get fewer tokens per wave, halved until they fit.  Every kernel here sizes
// its LDS regions and bounds its token and column loops by this count, so a
// wave simply leaves some of the 16 columns empty.
static DevPlan code_plan(const DevPlan& P)
{
    DevPlan C = P;
    while (C.wave_tokens > 1 && !code_rows_fit(C)) C.wave_tokens >>= 1;
    return C;
}

bool code_kernels_fit(const DevPlan& P)
{
    return code_rows_fit(code_plan(P));
}

// Kernel variants: index groups NG in {3, 4, 5, 6, 8} (a larger NG than the
// plan needs is exact: the extra table rows are zero) and the width of the
// leaf parents' sign bits.
int ng_variant(const DevPlan& P)
{
    return P.nt_groups <= 3 ? 3 : P.nt_groups <= 6 ? P.nt_groups : 8;
}

template <bool OB, int NG, bool PB>
static void launch_decode_v(const DevPlan& P, dim3 grid, size_t lds, hipStream_t stream, const int32_t* idx,
                            const float* coef, int64_t T, void* y)
{
    allow_lds(decode2_kernel<OB, NG, PB>, lds);
    hipLaunchKernelGGL((decode2_kernel<OB, NG, PB>), grid, dim3(kThreads), lds, stream, P, idx, coef, T, y);
}

template <bool OB, bool PB>
static void launch_decode_ng(const DevPlan& P, dim3 grid, size_t lds, hipStream_t stream, const int32_t* idx,
                             const float* coef, int64_t T, void* y)
{
    switch (ng_variant(P)) {
    case 3: launch_decode_v<OB, 3, PB>(P, grid, lds, stream, idx, coef, T, y); break;
    case 4: launch_decode_v<OB, 4, PB>(P, grid, lds, stream, idx, coef, T, y); break;
    case 5: launch_decode_v<OB, 5, PB>(P, grid, lds, stream, idx, coef, T, y); break;
    case 6: launch_decode_v<OB, 6, PB>(P, grid, lds, stream, idx, coef, T, y); break;
    default: launch_decode_v<OB, 8, PB>(P, grid, lds, stream, idx, coef, T, y); break;
    }
}

hipError_t launch_decode2(const DevPlan& Pp, const int32_t* idx, const float* coef, int64_t T, void* y, bool y_bf16,
                          hipStream_t stream)
{
    const DevPlan P = code_plan(Pp);
    const size_t lds = code_lds_bytes(P, false, true);
    if (lds > (size_t)kLdsBudget) return hipErrorInvalidValue;
    const dim3 grid = code_grid(P, T, lds, 1);
    const bool pb16 = P.pb_bytes == 2;
    if (y_bf16 && pb16) launch_decode_ng<true, true>(P, grid, lds, stream, idx, coef, T, y);
    else if (y_bf16) launch_decode_ng<true, false>(P, grid, lds, stream, idx, coef, T, y);
    else if (pb16) launch_decode_ng<false, true>(P, grid, lds, stream, idx, coef, T, y);
    else launch_decode_ng<false, false>(P, grid, lds, stream, idx, coef, T, y);
    return hipGetLastError();
}

struct BwdExtra {
    const float* gc;
    const void* gx;
    const float2* stats;
};

template <bool GB, bool XB, int NG, bool PB>
static void launch_bwd_v(const DevPlan& P, dim3 grid, size_t lds, hipStream_t stream, const int32_t* idx,
                         const void* g, int64_t T, float* gc, void* gx, BwdExtra ex)
{
    if constexpr (GB && XB) {
        if (P.wave_tokens == 1 && P.k_tot <= 256) {
            allow_lds(decode_bwd2_kernel<GB, XB, NG, PB, true>, lds);
            hipLaunchKernelGGL((decode_bwd2_kernel<GB, XB, NG, PB, true>), grid, dim3(kThreads), lds, stream, P, idx, g,
                               T, gc, gx, ex.gc, ex.gx, ex.stats);
            return;
        }
    }
    allow_lds(decode_bwd2_kernel<GB, XB, NG, PB>, lds);
    hipLaunchKernelGGL((decode_bwd2_kernel<GB, XB, NG, PB>), grid, dim3(kThreads), lds, stream, P, idx, g, T, gc, gx,
                       ex.gc, ex.gx, ex.stats);
}

template <bool GB, bool XB, bool PB>
static void launch_bwd_ng(const DevPlan& P, dim3 grid, size_t lds, hipStream_t stream, const int32_t* idx,
                          const void* g, int64_t T, float* gc, void* gx, BwdExtra ex)
{
    switch (ng_variant(P)) {
    case 3: launch_bwd_v<GB, XB, 3, PB>(P, grid, lds, stream, idx, g, T, gc, gx, ex); break;
    case 4: launch_bwd_v<GB, XB, 4, PB>(P, grid, lds, stream, idx, g, T, gc, gx, ex); break;
    case 5: launch_bwd_v<GB, XB, 5, PB>(P, grid, lds, stream, idx, g, T, gc, gx, ex); break;
    case 6: launch_bwd_v<GB, XB, 6, PB>(P, grid, lds, stream, idx, g, T, gc, gx, ex); break;
    default: launch_bwd_v<GB, XB, 8, PB>(P, grid, lds, stream, idx, g, T, gc, gx, ex); break;
    }
}

template <bool GB, bool XB>
static void launch_bwd_ub(const DevPlan& P, dim3 grid, size_t lds, hipStream_t stream, const int32_t* idx,
                          const void* g, int64_t T, float* gc, void* gx, BwdExtra ex)
{
    if (P.pb_bytes == 2) launch_bwd_ng<GB, XB, true>(P, grid, lds, stream, idx, g, T, gc, gx, ex);
    else launch_bwd_ng<GB, XB, false>(P, grid, lds, stream, idx, g, T, gc, gx, ex);
}

hipError_t launch_decode_bwd2(const DevPlan& Pp, const int32_t* idx, const void* g, bool g_bf16, int64_t T,
                              float* grad_coef, void* grad_x, bool gx_bf16, hipStream_t stream,
                              const float* add_grad_coef, const void* add_grad_x, const float* stats)
{
    const DevPlan P = code_plan(Pp);
    const size_t lds = code_lds_bytes(P, true, g_bf16);
    if (lds > (size_t)kLdsBudget) return hipErrorInvalidValue;
    const dim3 grid = code_grid(P, T, lds, 4);
    const BwdExtra ex{add_grad_coef, add_grad_x, (const float2*)stats};
    if (g_bf16 && gx_bf16) launch_bwd_ub<true, true>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x, ex);
    else if (g_bf16) launch_bwd_ub<true, false>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x, ex);
    else if (gx_bf16) launch_bwd_ub<false, true>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x, ex);
    else launch_bwd_ub<false, false>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x, ex);
    return hipGetLastError();
}

}  // namespace dpb
