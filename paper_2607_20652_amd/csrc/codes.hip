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
//  * backward: grad_coef of the children of a parent p is
//    Gamma_l (phi~_p (.) g) -- the encoder's child-scoring contraction with g
//    in place of x (§2.2 child-scoring equation) -- on the matrix cores; the
//    parent's sign pattern comes from nibble tables (parity is linear in the
//    index bits), and grad_x is the decode of grad_coef.
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
constexpr int kBatch = 8;  // column-decode fragments fetched per batch

struct Wave {
    int lane;
    int64_t t0;
    int ntok;
    int32_t* idx;     // [TPW][k]
    float* coef;      // [TPW][k]
    int32_t* route;   // [TPW][k]: (parent slot << 16) | j, or -1
    int32_t* dir;     // [TPW][k]: 1 when a slot is decoded directly
    int32_t* par;     // [16] parent index of each column row
    float* alpha;     // [16][dpad] column coefficients
    int32_t* claim;   // [16][dpad] lowest slot claiming (row, j)
    float* y;         // [TPW][dp] output accumulator (fp32)
    uint32_t* pairs;  // [TPW][dp/2] |g| as bf16 pairs in the paired coordinate order
    uint32_t* signw;  // [TPW][nchunk] sign bits of g, natural order
    float* gf;        // [TPW][dp] fp32 g (fp32 activations)
    uint32_t* cw;     // [16][nchunk] column sign bitmaps (g's sign folded in for bf16)
    float* score;     // [16][16] scores of one column block and generator tile
    const uint32_t* mask;  // [dp] row masks (shared)
    const int32_t* gtab;   // generator hash tables (shared)
    const uint32_t* gens;  // generators (shared)
    const uint32_t* nt;    // nibble tables (shared, backward only)
};

__device__ __forceinline__ int rdlane(int v, int l) { return __builtin_amdgcn_readlane(v, l); }

// Routes every hashed slot of levels >= lmin: finds the first parent slot q
// of the previous level (in slot order) and the generator j with
// c = parent_q XOR g_j, by looking c XOR parent_q up in the level's generator
// hash table.  W.route[tt][s] = (q << 16) | j, or -1 when no pair exists.
__device__ void route_slots(const DevPlan& P, const Wave& W, int lmin)
{
    const int k = P.k_tot, TPW = P.wave_tokens;
    for (int job = W.lane; job < TPW * k; job += 64) {
        const int tt = job / k, s = job - tt * k;
        int rt = -1;
        const int32_t c = W.idx[job];
        if (tt < W.ntok && c >= P.d && P.gtab_total > 0 && P.levels > 1 && s >= P.slot_base[lmin]) {
            int l = 1;
            while (l + 1 < P.levels && s >= P.slot_base[l + 1]) ++l;
            const int bits = P.gtab_bits[l], Kp = P.active[l - 1];
            const uint32_t hmask = (1u << bits) - 1u;
            const int32_t* tab = W.gtab + P.gtab_off[l];
            const uint32_t* gl = W.gens + P.gens_off[l];
            const int32_t* parents = W.idx + tt * k + P.slot_base[l - 1];
            for (int q = 0; q < Kp && rt < 0; ++q) {
                const int32_t p = parents[q];
                if (p < 0) continue;
                const uint32_t x = (uint32_t)c ^ (uint32_t)p;
                uint32_t h = (x * kGenHashMul) >> (32 - bits);
                for (int32_t j = tab[h]; j >= 0; h = (h + 1) & hmask, j = tab[h]) {
                    if (gl[j] == x) {
                        rt = (q << 16) | j;
                        break;
                    }
                }
            }
        }
        W.route[job] = rt;
    }
}

// Decode of the wave's tokens from W.idx and coefficients `cf` into W.y.
// W.route holds the routes of the last level's slots.
template <bool EXACT3, int UB>
__device__ void decode_tokens(const DevPlan& P, const Wave& W, const float* cf)
{
    const int k = P.k_tot, d = P.d, dp = P.dp, TPW = P.wave_tokens, lane = W.lane;
    const int L1 = P.levels - 1;
    const bool cols = P.leaf_columns != 0;

    if (cols) {
        const int Kc = P.active[L1 - 1], CPT = P.cpt[L1], KL = P.active[L1], dpad = P.dpad[L1];
        const int sbL = P.slot_base[L1], sbP = P.slot_base[L1 - 1];
        if (lane < 16) {
            const int tt = lane / CPT, q = lane % CPT;
            W.par[lane] = (tt < W.ntok && q < Kc) ? W.idx[tt * k + sbP + q] : -1;
        }
        for (int i = lane; i < 16 * dpad; i += 64) {
            W.alpha[i] = 0.f;
            W.claim[i] = 0x7FFFFFFF;
        }
        wave_sync();
        for (int tt = 0; tt < W.ntok; ++tt)
            for (int s = sbL + lane; s < sbL + KL; s += 64) {
                const int rt = W.route[tt * k + s];
                if (rt >= 0) atomicMin(&W.claim[(tt * CPT + (rt >> 16)) * dpad + (rt & 0xFFFF)], s);
            }
        wave_sync();
        for (int tt = 0; tt < W.ntok; ++tt)
            for (int s = sbL + lane; s < sbL + KL; s += 64) {
                const int rt = W.route[tt * k + s];
                const int at = rt >= 0 ? (tt * CPT + (rt >> 16)) * dpad + (rt & 0xFFFF) : 0;
                const bool mine = rt >= 0 && W.claim[at] == s;
                if (mine) W.alpha[at] = cf[tt * k + s];
                W.dir[tt * k + s] = mine ? 0 : 1;
            }
        wave_sync();

        // Gamma^T alpha on the matrix cores, then the parent's signs
        const int nkb = dpad / 16, row = lane & 15, grp = lane >> 4;
        bf16x4 ahi[4], amid[4], alo[4];
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
            uint32_t h[4] = {0, 0, 0, 0}, m[4] = {0, 0, 0, 0}, lo[4] = {0, 0, 0, 0};
            if (kb < nkb) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const float a = W.alpha[row * dpad + 16 * kb + 4 * grp + i];
                    if constexpr (EXACT3) {
                        split3(a, h[i], m[i], lo[i]);
                    } else {
                        h[i] = f32_to_bf16_rne(a);
                        lo[i] = f32_to_bf16_rne(a - bf16_bits_to_f32(h[i]));
                    }
                }
            }
            ahi[kb] = __builtin_bit_cast(bf16x4, (u32x2){h[0] | (h[1] << 16), h[2] | (h[3] << 16)});
            amid[kb] = __builtin_bit_cast(bf16x4, (u32x2){m[0] | (m[1] << 16), m[2] | (m[3] << 16)});
            alo[kb] = __builtin_bit_cast(bf16x4, (u32x2){lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16)});
        }
        uint32_t pr[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) pr[i] = (uint32_t)W.par[4 * grp + i];
        const u32x2* bfr = (const u32x2*)P.gamma_t + P.gamma_t_off[L1] + lane;
        const int tok = (4 * grp) / CPT;
        const bool writer = (grp % (CPT / 4)) == 0 && tok < TPW;
        const int ncb = dp / 16;
        for (int cb0 = 0; cb0 < ncb; cb0 += kBatch) {
            u32x2 bf[kBatch][4];
            uint32_t M[kBatch];
#pragma unroll
            for (int e = 0; e < kBatch; ++e) {
                const int cb = cb0 + e < ncb ? cb0 + e : ncb - 1;
#pragma unroll
                for (int kb = 0; kb < 4; ++kb)
                    if (kb < nkb) bf[e][kb] = bfr[((int64_t)cb * nkb + kb) * 64];
                M[e] = W.mask[16 * cb + row];
            }
#pragma unroll
            for (int e = 0; e < kBatch; ++e) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int kb = 0; kb < 4; ++kb) {
                    if (kb >= nkb) break;
                    const bf16x4 b = __builtin_bit_cast(bf16x4, bf[e][kb]);
                    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(ahi[kb], b, acc, 0, 0, 0);
                    if constexpr (EXACT3) acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(amid[kb], b, acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(alo[kb], b, acc, 0, 0, 0);
                }
                float v = signed_by_parity(acc[0], M[e] & pr[0]) + signed_by_parity(acc[1], M[e] & pr[1]) +
                          signed_by_parity(acc[2], M[e] & pr[2]) + signed_by_parity(acc[3], M[e] & pr[3]);
                if (CPT >= 8) v += __shfl_xor(v, 16, 64);
                if (CPT >= 16) v += __shfl_xor(v, 32, 64);
                if (writer && cb0 + e < ncb) W.y[tok * dp + 16 * (cb0 + e) + row] = v;
            }
        }
    } else {
        for (int i = lane; i < TPW * dp; i += 64) W.y[i] = 0.f;
    }
    wave_sync();

    // direct slots: +-coef at every coordinate; lanes own iota = lane + 64u.
    // Slot data sits in registers (lane s <-> slot s0 + s) and is broadcast.
    const int U = (dp + 63) / 64;
    const int sbL = P.slot_base[L1];
    for (int tt = 0; tt < W.ntok; ++tt) {
        float* yt = W.y + tt * dp;
        for (int u0 = 0; u0 < U; u0 += UB) {
            float acc[UB];
            uint32_t M[UB];
#pragma unroll
            for (int uu = 0; uu < UB; ++uu) {
                const int iota = lane + 64 * (u0 + uu);
                const bool ok = iota < dp;
                acc[uu] = ok ? yt[iota] : 0.f;
                M[uu] = ok ? W.mask[iota] : 0u;
            }
            for (int s0 = 0; s0 < k; s0 += 64) {
                const int s = s0 + lane;
                int32_t cv = s < k ? W.idx[tt * k + s] : -1;
                if (s < k && cols && s >= sbL && W.dir[tt * k + s] == 0) cv = -1;  // decoded through its column
                const int av = s < k ? __float_as_int(cf[tt * k + s]) : 0;
                uint64_t live = __ballot(cv >= d);
                while (live) {
                    const int b = __builtin_ctzll(live);
                    live &= live - 1;
                    const uint32_t c = (uint32_t)rdlane(cv, b);
                    const uint32_t au = (uint32_t)rdlane(av, b);
                    const uint32_t sg = au >> 31, mag = au & 0x7FFFFFFFu;
#pragma unroll
                    for (int uu = 0; uu < UB; ++uu)
                        acc[uu] += __uint_as_float(((__popc(M[uu] & c) + sg) << 31) | mag);
                }
            }
#pragma unroll
            for (int uu = 0; uu < UB; ++uu) {
                const int iota = lane + 64 * (u0 + uu);
                if (iota < dp) yt[iota] = P.rsd * acc[uu];
            }
        }
    }
    wave_sync();

    // basis slots: coefficient at their own coordinate, in slot order
    for (int tt = 0; tt < W.ntok; ++tt)
        for (int s0 = 0; s0 < k; s0 += 64) {
            const int s = s0 + lane;
            const int32_t c = s < k ? W.idx[tt * k + s] : -1;
            const int a = s < k ? __float_as_int(cf[tt * k + s]) : 0;
            uint64_t m = __ballot(c >= 0 && c < d);
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

__device__ Wave make_wave(const DevPlan& P, unsigned char* smem, bool scoring, bool act_bf16, int wave, int lane)
{
    const CodeLayout CL = code_layout(P, scoring, act_bf16);
    unsigned char* b = smem + code_shared_bytes(P, scoring) + (unsigned)wave * CL.bytes;
    Wave W;
    W.lane = lane;
    W.t0 = 0;
    W.ntok = 0;
    W.idx = (int32_t*)(b + CL.idx);
    W.coef = (float*)(b + CL.coef);
    W.route = (int32_t*)(b + CL.route);
    W.dir = (int32_t*)(b + CL.dir);
    W.par = (int32_t*)(b + CL.par);
    W.alpha = (float*)(b + CL.alpha);
    W.claim = (int32_t*)(b + CL.claim);
    W.y = (float*)(b + CL.y);
    W.pairs = (uint32_t*)(b + CL.pairs);
    W.signw = (uint32_t*)(b + CL.signw);
    W.gf = (float*)(b + CL.y);
    W.cw = (uint32_t*)(b + CL.cw);
    W.score = (float*)(b + CL.score);
    W.mask = (const uint32_t*)smem;
    W.gtab = (const int32_t*)(smem + align16u(P.dp * 4));
    W.gens = (const uint32_t*)(smem + align16u(P.dp * 4) + align16u(P.gtab_total * 4));
    W.nt = (const uint32_t*)(smem + align16u(P.dp * 4) + align16u(P.gtab_total * 4) + align16u(P.gens_total * 4));
    return W;
}

template <bool OUT_BF16>
__device__ void write_rows(const DevPlan& P, const Wave& W, void* out)
{
    for (int tt = 0; tt < W.ntok; ++tt)
        for (int iota = W.lane; iota < P.d; iota += 64)
            store_act<OUT_BF16>(out, (W.t0 + tt) * P.d + iota, W.y[tt * P.dp + iota]);
}

__device__ void load_shared(const DevPlan& P, unsigned char* smem, bool with_nt)
{
    uint32_t* s_mask = (uint32_t*)smem;
    int32_t* s_gtab = (int32_t*)(smem + align16u(P.dp * 4));
    uint32_t* s_gens = (uint32_t*)(smem + align16u(P.dp * 4) + align16u(P.gtab_total * 4));
    for (int i = threadIdx.x; i < P.dp; i += kThreads) s_mask[i] = P.masks[i];
    for (int i = threadIdx.x; i < P.gtab_total; i += kThreads) s_gtab[i] = P.gtab[i];
    for (int i = threadIdx.x; i < P.gens_total; i += kThreads) s_gens[i] = P.gens[i];
    if (with_nt) {
        uint32_t* s_nt = (uint32_t*)((unsigned char*)s_gens + align16u(P.gens_total * 4));
        for (int i = threadIdx.x; i < P.nt_groups * 16 * P.nchunk; i += kThreads) s_nt[i] = P.nt[i];
    }
    __syncthreads();
}

template <bool OUT_BF16, int UB>
__global__ __launch_bounds__(kThreads) void decode2_kernel(DevPlan P, const int32_t* __restrict__ idx,
                                                           const float* __restrict__ coef, int64_t T,
                                                           void* __restrict__ y)
{
    extern __shared__ __align__(16) unsigned char smem[];
    load_shared(P, smem, false);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, TPW = P.wave_tokens, k = P.k_tot;
    Wave W = make_wave(P, smem, false, true, wave, lane);
    const int64_t ngroups = (T + TPW - 1) / TPW;
    for (int64_t grp = (int64_t)blockIdx.x * kCodeWaves + wave; grp < ngroups;
         grp += (int64_t)gridDim.x * kCodeWaves) {
        W.t0 = grp * TPW;
        W.ntok = (int)min((int64_t)TPW, T - W.t0);
        for (int i = lane; i < TPW * k; i += 64) {
            const bool live = i / k < W.ntok;
            W.idx[i] = live ? idx[W.t0 * k + i] : -1;
            W.coef[i] = live ? coef[W.t0 * k + i] : 0.f;
            W.route[i] = -1;
            W.dir[i] = 1;
        }
        wave_sync();
        if (P.leaf_columns) {
            route_slots(P, W, P.levels - 1);
            wave_sync();
        }
        decode_tokens<!OUT_BF16, UB>(P, W, W.coef);
        write_rows<OUT_BF16>(P, W, y);
        wave_sync();
    }
}

// g at coordinate iota of token tt, from the LDS copy.
template <bool G_BF16>
__device__ __forceinline__ float g_at(const DevPlan& P, const Wave& W, int tt, int iota)
{
    if constexpr (G_BF16) return pair_value(P, W.pairs, W.signw, tt, iota);
    else return W.gf[tt * P.dp + iota];
}

// Child scores of the parent columns of level l against the wave's g,
// written to the coefficients of the slots routed to them.
template <bool G_BF16>
__device__ void score_level(const DevPlan& P, const Wave& W, int l)
{
    const int k = P.k_tot, TPW = P.wave_tokens, lane = W.lane;
    const int CPT = P.cpt[l], Kp = P.active[l - 1], Kl = P.active[l];
    const int ncol = TPW * CPT, NB = (ncol + 15) / 16, sbp = P.slot_base[l - 1], sbl = P.slot_base[l];
    const ActTile A{W.pairs, W.signw, W.gf};
    for (int nb = 0; nb < NB; ++nb) {
        column_bitmaps<G_BF16>(P, lane, W.ntok, l, nb, W.idx + sbp, k, Kp, A, W.nt, W.cw);
        wave_sync();
        const int col = lane & 15, kq = lane >> 4;
        const int r = nb * 16 + col, tt = r / CPT, q = r % CPT;
        const bool valid = r < ncol && tt < W.ntok && q < Kp && W.idx[tt * k + sbp + q] >= 0;
        const int trow = valid ? tt : 0;
        for (int mb = 0; mb < P.mblocks[l]; ++mb) {
            const f32x4 acc = mfma_scores<G_BF16>(P, lane, l, mb, valid, trow, A, W.cw);
#pragma unroll
            for (int i = 0; i < 4; ++i) W.score[col * 16 + kq * 4 + i] = acc[i] * P.rsd;
            wave_sync();
            // slots routed to a column of this block and a generator of this tile
            for (int tt2 = 0; tt2 < W.ntok; ++tt2)
                for (int s = sbl + lane; s < sbl + Kl; s += 64) {
                    const int rt = W.route[tt2 * k + s];
                    if (rt < 0) continue;
                    const int r2 = tt2 * CPT + (rt >> 16), j = rt & 0xFFFF;
                    if (r2 / 16 == nb && j / 16 == mb) W.coef[tt2 * k + s] = W.score[(r2 - nb * 16) * 16 + (j & 15)];
                }
            wave_sync();
        }
    }
}

template <bool G_BF16, bool GX_BF16, int UB>
__global__ __launch_bounds__(kThreads) void decode_bwd2_kernel(DevPlan P, const int32_t* __restrict__ idx,
                                                               const void* __restrict__ g, int64_t T,
                                                               float* __restrict__ grad_coef,
                                                               void* __restrict__ grad_x)
{
    extern __shared__ __align__(16) unsigned char smem[];
    load_shared(P, smem, true);
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, TPW = P.wave_tokens, k = P.k_tot;
    const int d = P.d, dp = P.dp;
    Wave W = make_wave(P, smem, true, G_BF16, wave, lane);
    const int64_t ngroups = (T + TPW - 1) / TPW;
    for (int64_t grp = (int64_t)blockIdx.x * kCodeWaves + wave; grp < ngroups;
         grp += (int64_t)gridDim.x * kCodeWaves) {
        const int64_t t0 = grp * TPW;
        W.t0 = t0;
        W.ntok = (int)min((int64_t)TPW, T - t0);

        // codes, routes reset, and g in LDS
        for (int i = lane; i < TPW * k; i += 64) {
            W.idx[i] = i / k < W.ntok ? idx[t0 * k + i] : -1;
            W.route[i] = -1;
            W.dir[i] = 1;
        }
        if constexpr (G_BF16) {
            load_pairs(P, lane, W.ntok, TPW, (const uint16_t*)g, t0, W.pairs, W.signw);
        } else {
            const float* gfp = (const float*)g;
            for (int e = lane; e < TPW * dp; e += 64) {
                const int tt = e / dp, iota = e - tt * dp;
                W.gf[e] = (tt < W.ntok && iota < d) ? gfp[(t0 + tt) * d + iota] : 0.f;
            }
        }
        wave_sync();

        // route every slot of levels >= 1 to a parent slot of the previous level
        route_slots(P, W, 1);
        // coefficients for basis slots and padding
        for (int job = lane; job < TPW * k; job += 64) {
            const int tt = job / k;
            const int32_t c = W.idx[job];
            float v = 0.f;
            if (tt < W.ntok && c >= 0 && c < d) v = g_at<G_BF16>(P, W, tt, c);
            W.coef[job] = v;
        }
        wave_sync();

        // grad_coef of routed slots: child scores of each parent column against g
        for (int l = 1; l < P.levels; ++l) score_level<G_BF16>(P, W, l);

        // hashed slots that route nowhere: a direct reduction over the coordinates
        for (int tt = 0; tt < W.ntok; ++tt)
            for (int s0 = 0; s0 < k; s0 += 64) {
                const int s = s0 + lane;
                const int32_t cs = s < k ? W.idx[tt * k + s] : -1;
                uint64_t todo = __ballot(s < k && cs >= d && W.route[tt * k + s] < 0);
                while (todo) {
                    const int b = __builtin_ctzll(todo);
                    todo &= todo - 1;
                    const uint32_t c = (uint32_t)rdlane(cs, b);
                    float part = 0.f;
                    for (int iota = lane; iota < d; iota += 64)
                        part += signed_by_parity(g_at<G_BF16>(P, W, tt, iota), W.mask[iota] & c);
                    const float sum = wave_sum(part);
                    if (lane == 0) W.coef[tt * k + s0 + b] = P.rsd * sum;
                }
            }
        wave_sync();
        for (int i = lane; i < W.ntok * k; i += 64) grad_coef[t0 * k + i] = W.coef[i];

        // grad_x = decode(idx, grad_coef); the scoring buffers are dead now
        decode_tokens<!GX_BF16, UB>(P, W, W.coef);
        write_rows<GX_BF16>(P, W, grad_x);
        wave_sync();
    }
}

int pick_ub(const DevPlan& P)
{
    const int U = (P.dp + 63) / 64;
    return U <= 4 ? 4 : U <= 8 ? 8 : U <= 12 ? 12 : 16;
}

size_t code_lds_bytes(const DevPlan& P, bool scoring, bool act_bf16)
{
    return code_shared_bytes(P, scoring) + (size_t)kCodeWaves * code_layout(P, scoring, act_bf16).bytes;
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

// Grid-stride launch: enough workgroups to fill the chip a few times over.
dim3 code_grid(const DevPlan& P, int64_t T, size_t lds)
{
    const int64_t groups = (T + P.wave_tokens - 1) / P.wave_tokens;
    const int64_t need = (groups + kCodeWaves - 1) / kCodeWaves;
    const int per_cu = lds ? (int)std::max<size_t>(1, (160 * 1024) / lds) : 4;
    const int64_t cap = (int64_t)device_cus() * std::min(per_cu, 8) * 4;
    return dim3((unsigned)std::max<int64_t>(1, std::min(need, cap)));
}

}  // namespace

bool code_kernels_fit(const DevPlan& P)
{
    return code_lds_bytes(P, true, true) <= (size_t)kLdsBudget && code_lds_bytes(P, true, false) <= (size_t)kLdsBudget;
}

#define DPB_DECODE_CASE(OB, UBV)                                                                          \
    do {                                                                                                  \
        allow_lds(decode2_kernel<OB, UBV>, lds);                                                          \
        hipLaunchKernelGGL((decode2_kernel<OB, UBV>), grid, dim3(kThreads), lds, stream, P, idx, coef, T, y); \
    } while (0)

hipError_t launch_decode2(const DevPlan& P, const int32_t* idx, const float* coef, int64_t T, void* y, bool y_bf16,
                          hipStream_t stream)
{
    const size_t lds = code_lds_bytes(P, false, true);
    if (lds > (size_t)kLdsBudget) return hipErrorInvalidValue;
    const dim3 grid = code_grid(P, T, lds);
    const int ub = pick_ub(P);
    if (y_bf16) {
        if (ub == 4) DPB_DECODE_CASE(true, 4);
        else if (ub == 8) DPB_DECODE_CASE(true, 8);
        else if (ub == 12) DPB_DECODE_CASE(true, 12);
        else DPB_DECODE_CASE(true, 16);
    } else {
        if (ub == 4) DPB_DECODE_CASE(false, 4);
        else if (ub == 8) DPB_DECODE_CASE(false, 8);
        else if (ub == 12) DPB_DECODE_CASE(false, 12);
        else DPB_DECODE_CASE(false, 16);
    }
    return hipGetLastError();
}

template <bool GB, bool XB>
static void launch_bwd_ub(const DevPlan& P, dim3 grid, size_t lds, hipStream_t stream, const int32_t* idx,
                          const void* g, int64_t T, float* gc, void* gx)
{
    const int ub = pick_ub(P);
    allow_lds(decode_bwd2_kernel<GB, XB, 4>, lds);
    allow_lds(decode_bwd2_kernel<GB, XB, 8>, lds);
    allow_lds(decode_bwd2_kernel<GB, XB, 12>, lds);
    allow_lds(decode_bwd2_kernel<GB, XB, 16>, lds);
    if (ub == 4)
        hipLaunchKernelGGL((decode_bwd2_kernel<GB, XB, 4>), grid, dim3(kThreads), lds, stream, P, idx, g, T, gc, gx);
    else if (ub == 8)
        hipLaunchKernelGGL((decode_bwd2_kernel<GB, XB, 8>), grid, dim3(kThreads), lds, stream, P, idx, g, T, gc, gx);
    else if (ub == 12)
        hipLaunchKernelGGL((decode_bwd2_kernel<GB, XB, 12>), grid, dim3(kThreads), lds, stream, P, idx, g, T, gc, gx);
    else
        hipLaunchKernelGGL((decode_bwd2_kernel<GB, XB, 16>), grid, dim3(kThreads), lds, stream, P, idx, g, T, gc, gx);
}

hipError_t launch_decode_bwd2(const DevPlan& P, const int32_t* idx, const void* g, bool g_bf16, int64_t T,
                              float* grad_coef, void* grad_x, bool gx_bf16, hipStream_t stream)
{
    const size_t lds = code_lds_bytes(P, true, g_bf16);
    if (lds > (size_t)kLdsBudget) return hipErrorInvalidValue;
    const dim3 grid = code_grid(P, T, lds);
    if (g_bf16 && gx_bf16) launch_bwd_ub<true, true>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x);
    else if (g_bf16) launch_bwd_ub<true, false>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x);
    else if (gx_bf16) launch_bwd_ub<false, true>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x);
    else launch_bwd_ub<false, false>(P, grid, lds, stream, idx, g, T, grad_coef, grad_x);
    return hipGetLastError();
}

}  // namespace dpb
