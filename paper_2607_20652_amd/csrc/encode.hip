// Encoder for gfx950: the top-down beam search of §2.2.
//
// A wave owns `wave_tokens` tokens (16 / CPT, CPT = parent columns per
// token rounded up to a power of two); their activations stay in LDS in the
// interleaved-halves layout of scoring.hpp.
//
//  * Level 0 (§2.1 Eq. 2: scoring a basis feature is a coordinate read):
//    each token's lanes take the maximum key over their coordinates; the
//    K_0-th largest lane maximum tau bounds the answer from below (the K_0
//    largest lane maxima are distinct keys >= tau), so only the few keys >= tau
//    are ranked exactly.  With bf16 activations a key is 32 bits: the bf16
//    magnitude above the complemented coordinate.
//  * With standardization statistics (mu, r = 1/sigma per feature, §2.2
//    "Score Standardization") every score s becomes z = (s - mu) r before it
//    is keyed: level 0 then uses 64-bit keys of fp32 z, and each child's
//    (mu, r) is gathered from the statistics table.
//  * Levels l >= 1: the children of every active parent are scored on the
//    matrix cores (§2.2 child-scoring equation); the 64-bit keys (|s| desc,
//    index asc, see device_common.hpp) are sorted by a bitonic network laid
//    over the MFMA output layout, unrolled at compile time, with DPP and
//    swizzle lane exchanges; a child reached from several parents has
//    bit-identical keys (same products, same reduction), so it appears as
//    adjacent duplicates and is kept once; the first K_l survivors are emitted
//    in order.
#include <algorithm>

#include "scoring.hpp"

namespace dpb {
namespace {

constexpr int kEncWaves = 4;
constexpr int kEncThreads = 64 * kEncWaves;

struct EncLayout {
    unsigned act, cw, par, list, cnt, bytes;
    int kmaxp;   // row stride of par
    int listn;   // keys per token in list
};

__host__ __device__ inline int pow2_ceil(int v)
{
    int p = 1;
    while (p < v) p <<= 1;
    return p;
}

__host__ __device__ inline int enc_r(const DevPlan& P)
{
    int mb = 1;
    for (int l = 1; l < P.levels; ++l) mb = P.mblocks[l] > mb ? P.mblocks[l] : mb;
    return 4 * pow2_ceil(mb);
}

__host__ __device__ inline EncLayout enc_layout(const DevPlan& P, bool act_bf16)
{
    EncLayout L;
    const int TPW = P.wave_tokens, LPT = 64 / TPW;
    const int ND = (P.dp / 2 + LPT - 1) / LPT;  // activation dwords per lane at level 0
    // level-0 candidates: the K_0 lanes whose maximum reaches tau, each with all its keys
    int listn = P.active[0] * (act_bf16 ? 2 * ND : (P.d + LPT - 1) / LPT);
    L.listn = listn;
    L.kmaxp = P.kmax;
    unsigned off = 0;
    L.act = off;
    off = align16u(off + (act_bf16 ? TPW * P.prow * 4 : TPW * P.dp * 4));
    L.cw = off;   off = align16u(off + 16 * P.cws * 4);
    L.par = off;  off = align16u(off + TPW * L.kmaxp * 4);
    L.list = off; off = align16u(off + TPW * listn * 8);
    L.cnt = off;  off = align16u(off + TPW * 4);
    L.bytes = off;
    return L;
}

// Shared LDS of an encoder workgroup: nibble tables, generators and, with
// standardization, the level-0 statistics.
__host__ __device__ inline unsigned enc_shared_bytes(const DevPlan& P, bool std)
{
    return align16u(P.nt_groups * 16 * P.nchunk * 4) + align16u(P.gens_total * 4) + (std ? align16u(P.d * 8) : 0u);
}

// Exchange with the lane whose index differs by m (a power of two): DPP for
// 1 and 2, swizzles up to 16, a permute for 32.
__device__ __forceinline__ uint32_t xlane(uint32_t v, int m, int x32addr)
{
    switch (m) {
    case 1: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
    case 2: return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
    case 4: return swz_xor<4>(v);
    case 8: return swz_xor<8>(v);
    case 16: return swz_xor<16>(v);
    default: return (uint32_t)__builtin_amdgcn_ds_bpermute(x32addr, (int)v);
    }
}

__device__ __forceinline__ uint64_t xlane64(uint64_t v, int m, int x32addr)
{
    return ((uint64_t)xlane((uint32_t)(v >> 32), m, x32addr) << 32) | xlane((uint32_t)v, m, x32addr);
}

template <typename K>
__device__ __forceinline__ K xlaneK(K v, int m, int x32addr)
{
    if constexpr (sizeof(K) == 8) return xlane64(v, m, x32addr);
    else return xlane(v, m, x32addr);
}

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src)
{
    const uint32_t hi = (uint32_t)__shfl((int)(v >> 32), src, 64);
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, 64);
    return ((uint64_t)hi << 32) | lo;
}

// Descending bitonic sort of one token's R * 2^NB keys: element e =
// lanepos * R + r lives in register r of the lane at position lanepos.  In
// the MFMA layout lanepos = q * 4 + kq (q = lane bits 0.., kq = lane bits
// 4, 5); otherwise lanepos bit b is lane bit b.  Every loop is unrolled, so
// the exchange pattern and the in-lane directions are compile-time constants.
template <int R, int NB, bool MFMA_LAYOUT, typename K>
__device__ __forceinline__ void sort_desc(K (&v)[R], int lanepos, int x32addr)
{
    constexpr int LR = R == 1 ? 0 : R == 2 ? 1 : R == 4 ? 2 : R == 8 ? 3 : 4;
#pragma unroll
    for (int ks = 1; ks <= LR + NB; ++ks) {
#pragma unroll
        for (int js = ks - 1; js >= 0; --js) {
            if (js >= LR) {
                const int b = js - LR;
                const int m = MFMA_LAYOUT ? (b < 2 ? (16 << b) : (1 << (b - 2))) : (1 << b);
                const bool up = (ks - LR < NB) && ((lanepos >> (ks - LR)) & 1);
                const bool lower = !((lanepos >> b) & 1);
                const bool tmax = lower != up;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const K o = xlaneK(v[r], m, x32addr);
                    const bool gt = o > v[r];
                    v[r] = (gt == tmax) ? o : v[r];
                }
            } else {
                const int j = 1 << js;
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    if (r & j) continue;
                    const bool up = (ks < LR) ? ((r >> ks) & 1) : ((ks - LR < NB) && ((lanepos >> (ks - LR)) & 1));
                    const K a = v[r], c = v[r | j];
                    const bool sw = up ? (a > c) : (a < c);
                    v[r] = sw ? c : a;
                    v[r | j] = sw ? a : c;
                }
            }
        }
    }
}

// Emits the first K distinct keys of each token straight from the sorted
// registers of the MFMA layout (position lanepos * R + r): duplicates are
// adjacent, the predecessor of register 0 comes from the lane at lanepos - 1,
// and ranks are prefix counts in lanepos order.  Writes slots [sb, sb + K)
// and records them as the next parents.
template <int R, int CPT>
__device__ __forceinline__ void emit_mfma(const DevPlan& P, const uint64_t (&key)[R], int lane, int lanepos, int ct,
                                          int prev_addr, uint64_t before_mask, uint64_t token_mask, int64_t t0,
                                          int ntok, int K, int sb, int32_t* par, int kmaxp, int32_t* out_idx,
                                          float* out_coef)
{
    const int k_tot = P.k_tot;
    const uint32_t ph = (uint32_t)__builtin_amdgcn_ds_bpermute(prev_addr, (int)(uint32_t)(key[R - 1] >> 32));
    const uint32_t pl = (uint32_t)__builtin_amdgcn_ds_bpermute(prev_addr, (int)(uint32_t)key[R - 1]);
    uint64_t prev = lanepos > 0 ? (((uint64_t)ph << 32) | pl) : 0ull;
    int kept = 0, cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool k = key[r] != 0ull && key[r] != prev;
        kept |= (int)k << r;
        cnt += (int)k;
        prev = key[r];
    }
    int before = 0, total = 0;
#pragma unroll
    for (int b = 0; b < 5; ++b) {
        const uint64_t m = __ballot((cnt >> b) & 1);
        before += (int)__popcll(m & before_mask) << b;
        total += (int)__popcll(m & token_mask) << b;
    }
    const bool live = ct < ntok;
    int rank = before;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (((kept >> r) & 1) && rank < K) {
            const uint32_t ci = key_index(key[r]);
            par[ct * kmaxp + rank] = (int32_t)ci;
            if (live) {
                out_idx[(t0 + ct) * k_tot + sb + rank] = (int32_t)ci;
                out_coef[(t0 + ct) * k_tot + sb + rank] = key_value(key[r]);
            }
        }
        rank += (kept >> r) & 1;
    }
    for (int r = total + lanepos; r < K; r += 4 * CPT) {
        par[ct * kmaxp + r] = -1;
        if (live) {
            out_idx[(t0 + ct) * k_tot + sb + r] = -1;
            out_coef[(t0 + ct) * k_tot + sb + r] = 0.f;
        }
    }
}

// Level 0, bf16 activations: 32-bit keys (|x| bf16 bits << 16 | 0xFFFF - iota).
// Lane li of token tt reads the interleaved dwords e = li + LPT m; dword e
// holds coordinates 32 (e >> 4) + (e & 15) (low half) and that + 16.
// Coordinates past d hold zeros, so their keys sort below every real key.
template <int LPT, int LLP>
__device__ void level0_bf16(const DevPlan& P, int lane, int64_t t0, int ntok, const uint32_t* pairs, uint64_t* list,
                            int listn, int* cnt, int32_t* par, int kmaxp, int32_t* out_idx, float* out_coef,
                            int x32addr)
{
    const int tt = lane >> LLP, li = lane & (LPT - 1), K0 = P.active[0], dp2 = P.dp / 2;
    const uint32_t* row = pairs + tt * P.prow;
    const int lo0 = 32 * (li >> 4) + (li & 15);  // coordinate of the low half of dword li
    constexpr uint32_t STEP = 2 * LPT;           // coordinate step per dword row
    uint32_t best = 0;
    {
        uint32_t c = 0xFFFFu - (uint32_t)lo0;
        for (int e = li; e < dp2; e += LPT, c -= STEP) {
            const uint32_t D = row[e];
            const uint32_t klo = ((D << 16) & 0x7FFF0000u) | c, khi = (D & 0x7FFF0000u) | (c - 16u);
            best = max(best, max(klo, khi));
        }
    }
    uint32_t sv[1] = {best};
    sort_desc<1, LLP, false>(sv, li, x32addr);
    const uint32_t tau = (uint32_t)__shfl((int)sv[0], (lane & ~(LPT - 1)) + K0 - 1, 64);
    if (li == 0) cnt[tt] = 0;
    wave_sync();
    uint32_t* lst = (uint32_t*)(list + tt * listn);
    {
        uint32_t c = 0xFFFFu - (uint32_t)lo0;
        for (int e = li; e < dp2; e += LPT, c -= STEP) {
            const uint32_t D = row[e];
            const uint32_t klo = ((D << 16) & 0x7FFF0000u) | c, khi = (D & 0x7FFF0000u) | (c - 16u);
            if (klo >= tau) lst[atomicAdd(&cnt[tt], 1)] = klo;
            if (khi >= tau) lst[atomicAdd(&cnt[tt], 1)] = khi;
        }
    }
    wave_sync();
    const int n = cnt[tt];
    const bool live = tt < ntok;
    for (int e = li; e < n; e += LPT) {
        const uint32_t ke = lst[e];
        int rank = 0;
        for (int f = 0; f < n; ++f) rank += lst[f] > ke;
        if (rank < K0) {
            const uint32_t iota = 0xFFFFu - (ke & 0xFFFFu);
            par[tt * kmaxp + rank] = (int32_t)iota;
            if (live) {
                out_idx[(t0 + tt) * P.k_tot + rank] = (int32_t)iota;
                out_coef[(t0 + tt) * P.k_tot + rank] = pair_value(P, pairs, tt, (int)iota);
            }
        }
    }
}

// Level 0, fp32 activations: 64-bit keys over natural-order coordinates.
template <int LPT, int LLP>
__device__ void level0_f32(const DevPlan& P, int lane, int64_t t0, int ntok, const float* xf, uint64_t* list,
                           int listn, int* cnt, int32_t* par, int kmaxp, int32_t* out_idx, float* out_coef,
                           int x32addr)
{
    const int tt = lane >> LLP, li = lane & (LPT - 1), K0 = P.active[0], d = P.d, dp = P.dp;
    const float* row = xf + tt * dp;
    uint64_t best = 0;
    for (int iota = li; iota < d; iota += LPT) best = max(best, make_key(row[iota], (uint32_t)iota));
    uint64_t sv[1] = {best};
    sort_desc<1, LLP, false>(sv, li, x32addr);
    const uint64_t tau = shfl_u64(sv[0], (lane & ~(LPT - 1)) + K0 - 1);
    if (li == 0) cnt[tt] = 0;
    wave_sync();
    uint64_t* lst = list + tt * listn;
    for (int iota = li; iota < d; iota += LPT) {
        const uint64_t kk = make_key(row[iota], (uint32_t)iota);
        if (kk >= tau) lst[atomicAdd(&cnt[tt], 1)] = kk;
    }
    wave_sync();
    const int n = cnt[tt];
    const bool live = tt < ntok;
    for (int e = li; e < n; e += LPT) {
        const uint64_t ke = lst[e];
        int rank = 0;
        for (int f = 0; f < n; ++f) rank += lst[f] > ke;
        if (rank < K0) {
            const uint32_t iota = key_index(ke);
            par[tt * kmaxp + rank] = (int32_t)iota;
            if (live) {
                out_idx[(t0 + tt) * P.k_tot + rank] = (int32_t)iota;
                out_coef[(t0 + tt) * P.k_tot + rank] = key_value(ke);
            }
        }
    }
}

// Level 0 on standardized scores z = (x - mu) r (§2.2 "Score
// Standardization"), in fp32: 64-bit keys over the coordinates, as level0_f32,
// with the level-0 statistics staged in LDS (st0).  With bf16 activations lane
// li reads the interleaved dwords e = li + LPT m (coordinates 32 (e >> 4) +
// (e & 15) and that + 16); coordinates past d get key 0.
template <int LPT, int LLP, bool X_BF16>
__device__ void level0_std(const DevPlan& P, int lane, int64_t t0, int ntok, const uint32_t* pairs, const float* xf,
                           const float2* st0, uint64_t* list, int listn, int* cnt, int32_t* par, int kmaxp,
                           int32_t* out_idx, float* out_coef, int x32addr)
{
    const int tt = lane >> LLP, li = lane & (LPT - 1), K0 = P.active[0], d = P.d;
    auto zkey = [&](float x, int iota) -> uint64_t {
        if (iota >= d) return 0ull;
        const float2 st = st0[iota];
        return make_key((x - st.x) * st.y, (uint32_t)iota);
    };
    uint64_t best = 0;
    if constexpr (X_BF16) {
        const uint32_t* row = pairs + tt * P.prow;
        for (int e = li; e < P.dp / 2; e += LPT) {
            const uint32_t D = row[e];
            const int lo = 32 * (e >> 4) + (e & 15);
            best = max(best, max(zkey(bf16_bits_to_f32(D & 0xFFFFu), lo), zkey(bf16_bits_to_f32(D >> 16), lo + 16)));
        }
    } else {
        const float* row = xf + tt * P.dp;
        for (int iota = li; iota < d; iota += LPT) best = max(best, zkey(row[iota], iota));
    }
    uint64_t sv[1] = {best};
    sort_desc<1, LLP, false>(sv, li, x32addr);
    const uint64_t tau = shfl_u64(sv[0], (lane & ~(LPT - 1)) + K0 - 1);
    if (li == 0) cnt[tt] = 0;
    wave_sync();
    uint64_t* lst = list + tt * listn;
    if constexpr (X_BF16) {
        const uint32_t* row = pairs + tt * P.prow;
        for (int e = li; e < P.dp / 2; e += LPT) {
            const uint32_t D = row[e];
            const int lo = 32 * (e >> 4) + (e & 15);
            const uint64_t klo = zkey(bf16_bits_to_f32(D & 0xFFFFu), lo), khi = zkey(bf16_bits_to_f32(D >> 16), lo + 16);
            if (klo >= tau && klo != 0ull) lst[atomicAdd(&cnt[tt], 1)] = klo;
            if (khi >= tau && khi != 0ull) lst[atomicAdd(&cnt[tt], 1)] = khi;
        }
    } else {
        const float* row = xf + tt * P.dp;
        for (int iota = li; iota < d; iota += LPT) {
            const uint64_t kk = zkey(row[iota], iota);
            if (kk >= tau) lst[atomicAdd(&cnt[tt], 1)] = kk;
        }
    }
    wave_sync();
    const int n = cnt[tt];
    const bool live = tt < ntok;
    for (int e = li; e < n; e += LPT) {
        const uint64_t ke = lst[e];
        int rank = 0;
        for (int f = 0; f < n; ++f) rank += lst[f] > ke;
        if (rank < K0) {
            const uint32_t iota = key_index(ke);
            par[tt * kmaxp + rank] = (int32_t)iota;
            if (live) {
                out_idx[(t0 + tt) * P.k_tot + rank] = (int32_t)iota;
                out_coef[(t0 + tt) * P.k_tot + rank] = key_value(ke);
            }
        }
    }
}

template <bool X_BF16, int CPT, int R, bool STD>
__global__ __launch_bounds__(kEncThreads) void encode3_kernel(DevPlan P, const void* __restrict__ xin, int64_t T,
                                                              const float2* __restrict__ stats,
                                                              int32_t* __restrict__ out_idx,
                                                              float* __restrict__ out_coef)
{
    constexpr int TPW = 16 / CPT, LPT = 64 / TPW;
    constexpr int CB = CPT == 4 ? 2 : CPT == 8 ? 3 : 4;  // log2 CPT
    constexpr int NB = CB + 2;                            // lane bits of a token in the MFMA layout
    constexpr int LLP = LPT == 16 ? 4 : LPT == 32 ? 5 : 6;
    extern __shared__ __align__(16) unsigned char smem[];
    uint32_t* s_nt = (uint32_t*)smem;
    uint32_t* s_gens = (uint32_t*)(smem + align16u(P.nt_groups * 16 * P.nchunk * 4));
    float2* s_st0 = (float2*)(smem + enc_shared_bytes(P, false));   // level-0 statistics (STD)
    for (int i = threadIdx.x; i < P.nt_groups * 16 * P.nchunk; i += kEncThreads) s_nt[i] = P.nt[i];
    for (int i = threadIdx.x; i < P.gens_total; i += kEncThreads) s_gens[i] = P.gens[i];
    if constexpr (STD)
        for (int i = threadIdx.x; i < P.d; i += kEncThreads) s_st0[i] = stats[i];
    __syncthreads();

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int d = P.d, dp = P.dp;
    const int x32 = (lane ^ 32) << 2;
    const EncLayout EL = enc_layout(P, X_BF16);
    unsigned char* wb = smem + enc_shared_bytes(P, STD) + (unsigned)wave * EL.bytes;
    uint32_t* pairs = (uint32_t*)(wb + EL.act);
    float* xf = (float*)(wb + EL.act);
    uint32_t* cw = (uint32_t*)(wb + EL.cw);
    int32_t* par = (int32_t*)(wb + EL.par);
    uint64_t* list = (uint64_t*)(wb + EL.list);
    int* cnt = (int*)(wb + EL.cnt);
    const ActTile A{pairs, xf};

    const int col = lane & 15, kq = lane >> 4, ct = col >> CB, q = col & (CPT - 1), lanepos = q * 4 + kq;
    // lanepos order inside a token: lanes of positions below mine, all lanes of my token, lane of lanepos - 1
    uint64_t before_mask = 0, token_mask = 0;
    for (int q2 = 0; q2 < CPT; ++q2)
        for (int k2 = 0; k2 < 4; ++k2) {
            const uint64_t bit = 1ull << (ct * CPT + q2 + 16 * k2);
            token_mask |= bit;
            if (q2 * 4 + k2 < lanepos) before_mask |= bit;
        }
    const int prev_addr = (kq > 0 ? lane - 16 : lane + 47) << 2;

    const int64_t ngroups = (T + TPW - 1) / TPW;
    for (int64_t grp = (int64_t)blockIdx.x * kEncWaves + wave; grp < ngroups;
         grp += (int64_t)gridDim.x * kEncWaves) {
        const int64_t t0 = grp * TPW;
        const int ntok = (int)min((int64_t)TPW, T - t0);

        if constexpr (X_BF16) {
            load_pairs(P, lane, ntok, TPW, (const uint16_t*)xin, t0, pairs);
        } else {
            const float* xs = (const float*)xin;
            for (int tt = 0; tt < TPW; ++tt)
                for (int iota = lane; iota < dp; iota += 64)
                    xf[tt * dp + iota] = (tt < ntok && iota < d) ? xs[(t0 + tt) * d + iota] : 0.f;
        }
        wave_sync();

        // ---- level 0
        if constexpr (STD)
            level0_std<LPT, LLP, X_BF16>(P, lane, t0, ntok, pairs, xf, s_st0, list, EL.listn, cnt, par, EL.kmaxp,
                                         out_idx, out_coef, x32);
        else if constexpr (X_BF16)
            level0_bf16<LPT, LLP>(P, lane, t0, ntok, pairs, list, EL.listn, cnt, par, EL.kmaxp, out_idx,
                                  out_coef, x32);
        else
            level0_f32<LPT, LLP>(P, lane, t0, ntok, xf, list, EL.listn, cnt, par, EL.kmaxp, out_idx, out_coef, x32);
        wave_sync();

        // ---- levels l >= 1
        for (int l = 1; l < P.levels; ++l) {
            const int Kp = P.active[l - 1], Dl = P.delta[l];
            column_bitmaps(P, lane, ntok, CB, 0, par, EL.kmaxp, Kp, s_nt, cw);
            wave_sync();
            const int32_t p = (ct < ntok && q < Kp) ? par[ct * EL.kmaxp + q] : -1;
            const bool valid = p >= 0;
            const int trow = valid ? ct : 0;
            const uint32_t* gens = s_gens + P.gens_off[l];
            // standardization statistics of this lane's children, requested
            // before the scoring so that the gathers overlap it
            float2 stv[R];
            if constexpr (STD) {
#pragma unroll
                for (int e = 0; e < R; ++e) {
                    const int j = 16 * (e >> 2) + 4 * kq + (e & 3);
                    stv[e] = (valid && j < Dl) ? stats[(uint32_t)p ^ gens[j]] : make_float2(0.f, 1.f);
                }
            }
            uint64_t keys[R];
#pragma unroll
            for (int mb = 0; mb < R / 4; ++mb) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                if (mb < P.mblocks[l]) acc = mfma_scores<X_BF16>(P, lane, l, mb, trow, A, cw);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = 16 * mb + 4 * kq + i;
                    const bool ok = valid && j < Dl;
                    const uint32_t c = ok ? (uint32_t)p ^ gens[j] : 0u;
                    float sc = acc[i] * P.rsd;
                    if constexpr (STD) sc = (sc - stv[4 * mb + i].x) * stv[4 * mb + i].y;
                    keys[4 * mb + i] = ok ? make_key(sc, c) : 0ull;
                }
            }
            sort_desc<R, NB, true>(keys, lanepos, x32);
            emit_mfma<R, CPT>(P, keys, lane, lanepos, ct, prev_addr, before_mask, token_mask, t0, ntok, P.active[l],
                              P.slot_base[l], par, EL.kmaxp, out_idx, out_coef);
            wave_sync();
        }
    }
}

}  // namespace

// Whether the standardized encoder's workgroup fits the LDS budget.
bool encode2_std_supported(const DevPlan& P)
{
    const size_t lds = enc_shared_bytes(P, true) + (size_t)kEncWaves * enc_layout(P, false).bytes;
    return encode2_supported(P) && lds <= (size_t)kLdsBudget;
}

bool encode2_supported(const DevPlan& P)
{
    const int TPW = P.wave_tokens, LPT = 64 / TPW;
    if (P.active[0] > LPT || enc_r(P) > 16 || P.d > 65535) return false;
    for (int l = 1; l < P.levels; ++l)
        if (P.cpt[l] > 16 || TPW * P.cpt[l] > 16) return false;
    if (16 / TPW != 4 && 16 / TPW != 8 && 16 / TPW != 16) return false;
    const size_t lds = enc_shared_bytes(P, false) + (size_t)kEncWaves * enc_layout(P, false).bytes;
    return lds <= (size_t)kLdsBudget;
}

hipError_t launch_encode2(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const float* stats, int32_t* idx,
                          float* coef, hipStream_t stream)
{
    const float2* st = (const float2*)stats;
    const size_t lds = enc_shared_bytes(P, stats != nullptr) + (size_t)kEncWaves * enc_layout(P, x_bf16).bytes;
    const int64_t groups = (T + P.wave_tokens - 1) / P.wave_tokens;
    const int64_t need = (groups + kEncWaves - 1) / kEncWaves;
    int cus = 256, dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
        cus = prop.multiProcessorCount;
    const int per_cu = (int)std::max<size_t>(1, (160 * 1024) / std::max<size_t>(lds, 1));
    const dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, (int64_t)cus * std::min(per_cu, 8) * 4)));
    const int R = enc_r(P), CPT = 16 / P.wave_tokens;
#define DPB_ENC(XB, CV, RV)                                                                                        \
    do {                                                                                                           \
        if (st) {                                                                                                  \
            allow_lds(encode3_kernel<XB, CV, RV, true>, lds);                                                      \
            hipLaunchKernelGGL((encode3_kernel<XB, CV, RV, true>), grid, dim3(kEncThreads), lds, stream, P, x, T,  \
                               st, idx, coef);                                                                     \
        } else {                                                                                                   \
            allow_lds(encode3_kernel<XB, CV, RV, false>, lds);                                                     \
            hipLaunchKernelGGL((encode3_kernel<XB, CV, RV, false>), grid, dim3(kEncThreads), lds, stream, P, x, T, \
                               st, idx, coef);                                                                     \
        }                                                                                                          \
    } while (0)
#define DPB_ENC_R(XB, CV)                    \
    do {                                     \
        if (R == 4) DPB_ENC(XB, CV, 4);      \
        else if (R == 8) DPB_ENC(XB, CV, 8); \
        else DPB_ENC(XB, CV, 16);            \
    } while (0)
    if (x_bf16) {
        if (CPT == 4) DPB_ENC_R(true, 4);
        else if (CPT == 8) DPB_ENC_R(true, 8);
        else DPB_ENC_R(true, 16);
    } else {
        if (CPT == 4) DPB_ENC_R(false, 4);
        else if (CPT == 8) DPB_ENC_R(false, 8);
        else DPB_ENC_R(false, 16);
    }
#undef DPB_ENC_R
#undef DPB_ENC
    return hipGetLastError();
}

}  // namespace dpb
