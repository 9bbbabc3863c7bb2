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
#include <mutex>

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

__host__ __device__ inline EncLayout enc_layout(const DevPlan& P, bool act_bf16, bool std = false)
{
    EncLayout L;
    const int TPW = P.wave_tokens, LPT = 64 / TPW;
    const int ND = (P.dp / 2 + LPT - 1) / LPT;  // activation dwords per lane at level 0
    // level-0 candidates: the K_0 lanes whose maximum reaches tau, each with all
    // its keys; listn counts 64-bit words per token.  Plain bf16 keys are 32
    // bits (2 ND per lane, two to a word); standardized and fp32 keys are 64.
    const int listn = (act_bf16 && !std) ? P.active[0] * ND
                                         : P.active[0] * (act_bf16 ? 2 * ND : (P.d + LPT - 1) / LPT);
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
// 1 and 2, swizzles up to 16, a permute for 32 (the LDS-path exchanges cost
// no vector-ALU slots, which the encoder is short of).
__device__ __forceinline__ uint32_t xlane(uint32_t v, int m, int x32addr)
{
    switch (m) {
    case 1: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
    case 2: return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
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
    (void)lane;
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

// The variants for bf16 input with one block of sixteen parent columns per
// level and plain scores (one or two tokens per wave) are held to 128
// registers, four waves per SIMD: both fit without spilling.  The two-token
// variant gains from it only because its level-0 list holds 32-bit keys at
// half the 64-bit size, so that four workgroups fit the LDS of a CU.
template <bool X_BF16, int CPT, int R, bool STD>
__global__ __launch_bounds__(kEncThreads, (X_BF16 && (CPT == 16 || CPT == 8) && R == 4 && !STD) ? 4 : 1) void encode3_kernel(DevPlan P, const void* __restrict__ xin, int64_t T,
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
    const EncLayout EL = enc_layout(P, X_BF16, STD);
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
    const int64_t gstride = (int64_t)gridDim.x * kEncWaves;
    // bf16 rows of two tokens with d <= 1024 (d a multiple of 8): the next
    // group's rows are requested while this group is encoded
    const bool pf = X_BF16 && TPW == 2 && d <= 1024 && (d & 7) == 0;
    u32x4 nx[4];
    auto fetch = [&](int64_t gp) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const int tt = e >> 1, o = (e & 1) * 512 + lane * 8;
            const int64_t t = gp * TPW + tt;
            nx[e] = (o < d && t < T) ? *(const u32x4*)((const uint16_t*)xin + t * d + o) : u32x4{0u, 0u, 0u, 0u};
        }
    };
    int64_t grp = (int64_t)blockIdx.x * kEncWaves + wave;
    if (pf && grp < ngroups) fetch(grp);
    for (; grp < ngroups; grp += gstride) {
        const int64_t t0 = grp * TPW;
        const int ntok = (int)min((int64_t)TPW, T - t0);

        if (pf) {
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int o = (e & 1) * 512 + lane * 8;
                if (o < dp) store_pair_piece(lane, nx[e], o, pairs + (e >> 1) * P.prow);
            }
            if (grp + gstride < ngroups) fetch(grp + gstride);
        } else if constexpr (X_BF16) {
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
            // standardization statistics of this lane's children, gathered
            // during the last batch of the first tile's scoring (read
            // unconditionally at an index that is always a feature: a
            // generator of the level when there is no parent)
            float2 stv[R];
            auto gather = [&]() {
                if constexpr (STD) {
#pragma unroll
                    for (int e = 0; e < R; ++e) {
                        const int j = 16 * (e >> 2) + 4 * kq + (e & 3);
                        const float2 v = stats[(valid ? (uint32_t)p : 0u) ^ gens[min(j, Dl - 1)]];
                        stv[e] = (valid && j < Dl) ? v : make_float2(0.f, 1.f);
                    }
                }
            };
            uint64_t keys[R];
#pragma unroll
            for (int mb = 0; mb < R / 4; ++mb) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                // batches of 6 chunks: faster here than 4, 8 or 12
                if (mb == 0) acc = mfma_scores<X_BF16, 6>(P, lane, l, mb, trow, A, cw, gather);
                else if (mb < P.mblocks[l]) acc = mfma_scores<X_BF16, 6>(P, lane, l, mb, trow, A, cw);
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
            // Levels that keep few of their candidates (K_l <= 2 CPT, the beam
            // levels): the K_l-th largest distinct lane maximum tau bounds the
            // answer (at least K_l distinct keys reach it), only the keys >= tau
            // are listed, and that short list (one key per lane of the token) is
            // sorted and emitted.  A token with more keys >= tau than lanes, or
            // any other level, sorts all its keys.
            const int Kl = P.active[l];
            bool done = false;
            if (Kl <= 2 * CPT && EL.listn >= 4 * CPT) {
                // the lane maxima are sorted by their magnitude word alone:
                // K_l distinct magnitudes at or above tau are K_l distinct
                // children, so tau = (that magnitude, lowest low word) still
                // admits the K_l largest keys (a valid key of magnitude 0
                // counts as none: then tau = 1)
                uint64_t m64 = keys[0];
#pragma unroll
                for (int r = 1; r < R; ++r) m64 = keys[r] > m64 ? keys[r] : m64;
                uint32_t mx[1] = {(uint32_t)(m64 >> 32)};
                sort_desc<1, NB, true>(mx, lanepos, x32);
                const uint32_t ph = (uint32_t)__builtin_amdgcn_ds_bpermute(prev_addr, (int)mx[0]);
                const uint32_t prev = lanepos > 0 ? ph : 0u;
                const bool kept = mx[0] != 0u && mx[0] != prev;
                const int rank = (int)__popcll(__ballot(kept) & before_mask);
                const uint64_t owner = __ballot(kept && rank == Kl - 1) & token_mask;
                uint64_t tau = 1ull;   // fewer than K_l distinct maxima: every key
                if (owner) {
                    const int oa = (int)__builtin_ctzll(owner) << 2;
                    tau = (uint64_t)(uint32_t)__builtin_amdgcn_ds_bpermute(oa, (int)mx[0]) << 32;
                }
                int c = 0;
#pragma unroll
                for (int r = 0; r < R; ++r) c += (int)(keys[r] >= tau);
                // c <= R keys per lane (R = 4, 8 or 16): 3, 4 or 5 count bits
                constexpr int CBITS = R <= 4 ? 3 : R <= 8 ? 4 : 5;
                int before = 0, total = 0;
#pragma unroll
                for (int b = 0; b < CBITS; ++b) {
                    const uint64_t m = __ballot((c >> b) & 1);
                    before += (int)__popcll(m & before_mask) << b;
                    total += (int)__popcll(m & token_mask) << b;
                }
                if (!__ballot(total > 4 * CPT)) {
                    uint64_t* tl = list + ct * EL.listn;
                    int pos = before;
#pragma unroll
                    for (int r = 0; r < R; ++r)
                        if (keys[r] >= tau) tl[pos++] = keys[r];
                    wave_sync();
                    uint64_t one[1] = {lanepos < total ? tl[lanepos] : 0ull};
                    wave_sync();
                    sort_desc<1, NB, true>(one, lanepos, x32);
                    emit_mfma<1, CPT>(P, one, lane, lanepos, ct, prev_addr, before_mask, token_mask, t0, ntok, Kl,
                                      P.slot_base[l], par, EL.kmaxp, out_idx, out_coef);
                    done = true;
                }
            }
            if (!done) {
                sort_desc<R, NB, true>(keys, lanepos, x32);
                emit_mfma<R, CPT>(P, keys, lane, lanepos, ct, prev_addr, before_mask, token_mask, t0, ntok, Kl,
                                  P.slot_base[l], par, EL.kmaxp, out_idx, out_coef);
            }
            wave_sync();
        }
    }
}

// ---------------------------------------------------------------------------
// Wide encoder: levels that score many children per parent (the paper's own
// hierarchies score 256, App. G Table 6).  Level 0 runs one wave per token.
// Each level l >= 1 is then a GEMM and a selection over chunks of tokens:
//  * wide_gemm_kernel: the scores of all K_{l-1} x Delta_l children of the
//    chunk's tokens, S[(t, q)][j] = <gamma_j, phi~_{p_tq} (.) x_t> (§2.2
//    child-scoring equation), as 16x16x32 bf16 MFMAs over a workgroup tile of
//    all generator rows x 128 (token, parent) columns.  A fragments (exact
//    +-1) are built from per-generator sign bitmaps held in LDS, B fragments
//    from the token rows and the parents' sign bitmaps (nibble tables), as in
//    the narrow encoder.  Its epilogue computes each token's threshold (the
//    K_l-th largest distinct magnitude among the lanes' maxima; distinct
//    magnitudes are distinct children) and writes only the (candidate, z)
//    entries at or above it to the workspace (with standardization it first
//    takes z = (s - mu) r with each candidate's gathered statistics); tokens
//    with too many entries and shapes it does not cover get the full scores.
//  * wide_select_kernel: one wave per token; AbsTopK with deduplication (a
//    child reached from several parents has bit-identical keys): the listed
//    entries, or the candidates above the same threshold found from the full
//    scores, are sorted as 64-bit keys by a bitonic network and the first K
//    distinct ones emitted; too many hits fall back to an exact extraction
//    (K rounds of a wave maximum below the previous key).
constexpr int kWideCols = 128;     // (token, parent) columns of a GEMM workgroup
constexpr int kWideList = 1024;    // collected keys per token
constexpr int kSeg = 16;           // keys per lane segment (64 kSeg = kWideList)
constexpr int kSegStride = kSeg + 1;
static_assert(64 * kSeg == kWideList && kSeg < 32, "segments fill the list; counts fit five bits");
constexpr int kWideThreads = 256;
static_assert(kWideThreads % kWideCols == 0, "column bitmaps: whole columns per thread group");
// (the fused epilogue keeps a lane's hits of one column tile, 4 MT <= 32 values, in one word)

template <bool X_BF16, bool STD>
__global__ __launch_bounds__(kWideThreads) void wide_level0_kernel(DevPlan P, const void* __restrict__ xin, int64_t T,
                                                                   const float2* __restrict__ stats,
                                                                   int32_t* __restrict__ out_idx,
                                                                   float* __restrict__ out_coef)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, d = P.d, dp = P.dp;
    const int ND = (dp / 2 + 63) / 64;
    const int listn = P.active[0] * (X_BF16 ? 2 * ND : (d + 63) / 64);
    const unsigned act_b = align16u(X_BF16 ? P.prow * 4 : dp * 4);
    const unsigned per_wave = act_b + align16u(listn * 8) + align16u((P.active[0] + 1) * 4) + 16;
    float2* st0 = (float2*)smem;
    unsigned char* wb = smem + (STD ? align16u(d * 8) : 0u) + wave * per_wave;
    uint32_t* pairs = (uint32_t*)wb;
    float* xf = (float*)wb;
    uint64_t* list = (uint64_t*)(wb + act_b);
    int32_t* par = (int32_t*)(wb + act_b + align16u(listn * 8));
    int* cnt = (int*)(wb + act_b + align16u(listn * 8) + align16u((P.active[0] + 1) * 4));
    if constexpr (STD) {
        for (int i = threadIdx.x; i < d; i += kWideThreads) st0[i] = stats[i];
        __syncthreads();
    }
    const int x32 = (lane ^ 32) << 2;
    for (int64_t t = (int64_t)blockIdx.x * 4 + wave; t < T; t += (int64_t)gridDim.x * 4) {
        if constexpr (X_BF16) {
            load_pairs(P, lane, 1, 1, (const uint16_t*)xin, t, pairs);
        } else {
            const float* xs = (const float*)xin;
            for (int iota = lane; iota < dp; iota += 64) xf[iota] = iota < d ? xs[t * d + iota] : 0.f;
        }
        wave_sync();
        if constexpr (STD)
            level0_std<64, 6, X_BF16>(P, lane, t, 1, pairs, xf, st0, list, listn, cnt, par, 0, out_idx, out_coef, x32);
        else if constexpr (X_BF16)
            level0_bf16<64, 6>(P, lane, t, 1, pairs, list, listn, cnt, par, 0, out_idx, out_coef, x32);
        else
            level0_f32<64, 6>(P, lane, t, 1, xf, list, listn, cnt, par, 0, out_idx, out_coef, x32);
        wave_sync();
    }
}

// Exclusive prefix over the wave of per-lane counts below 2^BITS.
template <int BITS>
__device__ __forceinline__ int wave_prefix(int cnt, int lane, int& total)
{
    const uint64_t below = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int before = 0;
    total = 0;
#pragma unroll
    for (int b = 0; b < BITS; ++b) {
        const uint64_t m = __ballot((cnt >> b) & 1);
        before += (int)__popcll(m & below) << b;
        total += (int)__popcll(m) << b;
    }
    return before;
}
__device__ __forceinline__ int wave_prefix5(int cnt, int lane, int& total) { return wave_prefix<5>(cnt, lane, total); }

// LDS of a GEMM workgroup: generator bitmaps, the tokens' rows, column bitmaps.
__host__ __device__ inline unsigned wide_gemm_lds(const DevPlan& P, int l, bool x_bf16)
{
    const int TT = kWideCols / P.cpt[l];
    return align16u(P.gpad[l] * P.cws * 4) + align16u(TT * (x_bf16 ? P.prow : P.dp) * 4) +
           align16u(kWideCols * P.cws * 4) + align16u(kWideCols * 4);
}

// Whether level l's GEMM selects in its epilogue: 16 to 64 parent columns per
// token (whole tokens per 64-column wave tile) and a token's score region can
// hold the kWideList (candidate, z) entries plus the discard entry after them.
// The fused epilogue reuses the staging LDS: the lane maxima, thresholds and
// counts below kWideEpiZ, then each wave's z values of one column tile.
constexpr unsigned kWideEpiZ = 8192;
__host__ __device__ inline unsigned wide_epi_lds(int MT) { return kWideEpiZ + 4u * 64u * (4u * MT + 4u) * 4u; }

__host__ __device__ inline bool wide_fused(const DevPlan& P, int l)
{
    const int MT = (P.delta[l] > 32 ? P.delta[l] : 32) / 32;
    return P.cpt[l] >= 16 && P.cpt[l] <= 64 && P.active[l - 1] * P.delta[l] >= 2 * (kWideList + 1) &&
           wide_gemm_lds(P, l, true) - align16u(kWideCols * 4) >= wide_epi_lds(MT);
}

// Scores of tokens [t0 + TT blockIdx.x, ...) of a chunk of ntok tokens at level
// l into scores[(t - t0) K_{l-1} + q][j] (t0-relative tokens).  MT = 16-row
// tiles per wave: waves (wr, wc) cover rows 16 MT wr .. and columns 64 wc ..
// FUSE: instead of all scores, each token's region receives the (candidate,
// z) entries at or above a threshold tau computed here from the lanes'
// largest magnitude keys (the selection's first pass), and counts[t - t0]
// their number; a token with more than kWideList entries gets its full scores
// and its count says so.  STD (with FUSE): every score is standardized here,
// z = (s - mu) r with the candidate's statistics (§2.2 "Score
// Standardization"), so that the threshold, the lists and any full scores
// hold z.
template <bool X_BF16, int MT, bool FUSE, bool STD>
__global__ __launch_bounds__(kWideThreads) __attribute__((amdgpu_waves_per_eu(2))) void wide_gemm_kernel(DevPlan P, int l, const void* __restrict__ xin,
                                                                 int64_t t0, int64_t ntok,
                                                                 const int32_t* __restrict__ idx,
                                                                 const float2* __restrict__ stats,
                                                                 float* __restrict__ scores,
                                                                 int* __restrict__ counts)
{
    static_assert(FUSE || !STD, "standardized scores only with the fused epilogue");
    extern __shared__ __align__(16) unsigned char smem[];
    const int KP = P.active[l - 1], KC = P.cpt[l], D = P.delta[l], nchunk = P.nchunk, d = P.d, dp = P.dp;
    const int csh = P.cpt_shift[l];   // KC = 2^csh
    const int TT = kWideCols >> csh;
    const int64_t tb = (int64_t)blockIdx.x * TT;
    const int nt_tok = (int)min((int64_t)TT, ntok - tb);
    uint32_t* s_gb = (uint32_t*)smem;   // row stride cws (odd): the 16 rows of a fragment on 16 banks
    unsigned char* p1 = smem + align16u(P.gpad[l] * P.cws * 4);
    uint32_t* pairs = (uint32_t*)p1;
    float* xf = (float*)p1;
    uint32_t* cw = (uint32_t*)(p1 + align16u(TT * (X_BF16 ? P.prow : dp) * 4));
    int32_t* s_pidx = (int32_t*)((unsigned char*)cw + align16u(kWideCols * P.cws * 4));   // parent of each column
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    {   // generator bitmaps: already in the LDS layout (row stride cws), 16-byte copies
        const u32x4* gsrc = (const u32x4*)(P.gbits + P.gbits_off[l]);
        u32x4* gdst = (u32x4*)s_gb;
        for (int i = threadIdx.x; i < P.gpad[l] * P.cws / 4; i += kWideThreads) gdst[i] = gsrc[i];
    }
    for (int tt = wave; tt < TT; tt += 4) {
        if constexpr (X_BF16) {
            load_pairs(P, lane, tt < nt_tok ? 1 : 0, 1, (const uint16_t*)xin, t0 + tb + tt, pairs + tt * P.prow);
        } else {
            const float* xs = (const float*)xin;
            for (int iota = lane; iota < dp; iota += 64)
                xf[tt * dp + iota] = (tt < nt_tok && iota < d) ? xs[(t0 + tb + tt) * d + iota] : 0.f;
        }
    }
    // parents' sign bitmaps: one nibble-table word per 4-bit group of the index;
    // lanes take consecutive columns of one word, so a table read touches one
    // 64-byte row of the table
    {
        const int col = threadIdx.x & (kWideCols - 1), tt = col >> csh, q = col & (KC - 1);
        const int32_t p = (tt < nt_tok && q < KP) ? idx[(t0 + tb + tt) * P.k_tot + P.slot_base[l - 1] + q] : -1;
        if (threadIdx.x < kWideCols) s_pidx[col] = p;
        // all kNtGroupsPadded groups are read (zero words past nt_groups): the
        // loads of a word are independent and wait once
        const uint32_t pu = p >= 0 ? (uint32_t)p : 0u;
        uint32_t toff[kNtGroupsPadded];
#pragma unroll
        for (int g = 0; g < kNtGroupsPadded; ++g) toff[g] = 4u * ((uint32_t)(g * nchunk * 16) + ((pu >> (4 * g)) & 15u));
        const unsigned char* ntb = (const unsigned char*)P.nt;
#pragma unroll 2
        for (int w = threadIdx.x / kWideCols; w < nchunk; w += kWideThreads / kWideCols) {
            uint32_t word = 0;
#pragma unroll
            for (int g = 0; g < kNtGroupsPadded; ++g) word ^= *(const uint32_t*)(ntb + toff[g] + (uint32_t)w * 64u);
            cw[col * P.cws + w] = p >= 0 ? word : 0u;
        }
    }
    __syncthreads();

    const int wr = wave >> 1, wc = wave & 1, c16 = lane & 15, kq = lane >> 4;
    f32x4 acc[MT][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int n = 0; n < 4; ++n) acc[mt][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    const int rowbase = wr * 16 * MT + c16;
    int bcol[4], btok[4];
#pragma unroll
    for (int n = 0; n < 4; ++n) {
        bcol[n] = wc * 64 + n * 16 + c16;
        btok[n] = bcol[n] >> csh;
    }
    // the LDS words of chunk c + 1 are requested before chunk c is computed
    // (two register sets, used in turn)
    struct Words {
        uint32_t a[MT], b[4];
        u32x4 pd[4];
    };
    auto fetch = [&](int c, Words& W) {
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) W.a[mt] = s_gb[(rowbase + 16 * mt) * P.cws + c];
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            W.b[n] = cw[bcol[n] * P.cws + c];
            if constexpr (X_BF16) W.pd[n] = *(const u32x4*)(pairs + btok[n] * P.prow + c * 16 + kq * 4);
        }
    };
    // A dword i: bf16 +-1 pair with the signs at coordinates 4kq + i and 16 + 4kq + i of the chunk
    auto afrag = [&](uint32_t w) -> bf16x8 {
        const uint32_t R = rotl32(w, 15u - 4u * (uint32_t)kq);
        u32x4 a;
        a.x = __builtin_amdgcn_bitop3_b32(R, 0x80008000u, 0x3F803F80u, 0xEA);   // (R & M) | one
        a.y = __builtin_amdgcn_bitop3_b32(__builtin_amdgcn_alignbit(R, R, 1), 0x80008000u, 0x3F803F80u, 0xEA);
        a.z = __builtin_amdgcn_bitop3_b32(__builtin_amdgcn_alignbit(R, R, 2), 0x80008000u, 0x3F803F80u, 0xEA);
        a.w = __builtin_amdgcn_bitop3_b32(__builtin_amdgcn_alignbit(R, R, 3), 0x80008000u, 0x3F803F80u, 0xEA);
        return __builtin_bit_cast(bf16x8, a);
    };
    auto compute = [&](int c, const Words& W) {
        if constexpr (X_BF16) {
            u32x4 b[4];
#pragma unroll
            for (int n = 0; n < 4; ++n) {
                const uint32_t R = rotl32(W.b[n], 15u - 4u * (uint32_t)kq);
                const u32x4 pd = W.pd[n];
                b[n].x = pd.x ^ (R & 0x80008000u);
                b[n].y = pd.y ^ (__builtin_amdgcn_alignbit(R, R, 1) & 0x80008000u);
                b[n].z = pd.z ^ (__builtin_amdgcn_alignbit(R, R, 2) & 0x80008000u);
                b[n].w = pd.w ^ (__builtin_amdgcn_alignbit(R, R, 3) & 0x80008000u);
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bf16x8 av = afrag(W.a[mt]);
#pragma unroll
                for (int n = 0; n < 4; ++n)
                    acc[mt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, b[n]), acc[mt][n],
                                                                         0, 0, 0);
            }
        } else {
            // fp32 activations: each value split exactly into three bf16 terms
            u32x4 bh[4], bm[4], bl[4];
#pragma unroll
            for (int n = 0; n < 4; ++n) {
                const int tt = btok[n];
                const uint32_t wd = W.b[n];
                uint32_t hi[8], mi[8], lo[8];
#pragma unroll
                for (int x = 0; x < 8; ++x) {
                    const int off = 4 * kq + (x >> 1) + 16 * (x & 1);
                    float v = xf[tt * dp + 32 * c + off];
                    v = __uint_as_float(__float_as_uint(v) ^ (((wd >> off) & 1u) << 31));
                    split3(v, hi[x], mi[x], lo[x]);
                }
                bh[n] = u32x4{hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16), hi[4] | (hi[5] << 16), hi[6] | (hi[7] << 16)};
                bm[n] = u32x4{mi[0] | (mi[1] << 16), mi[2] | (mi[3] << 16), mi[4] | (mi[5] << 16), mi[6] | (mi[7] << 16)};
                bl[n] = u32x4{lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16), lo[4] | (lo[5] << 16), lo[6] | (lo[7] << 16)};
            }
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bf16x8 av = afrag(W.a[mt]);
#pragma unroll
                for (int n = 0; n < 4; ++n) {
                    acc[mt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bh[n]),
                                                                         acc[mt][n], 0, 0, 0);
                    acc[mt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bm[n]),
                                                                         acc[mt][n], 0, 0, 0);
                    acc[mt][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bl[n]),
                                                                         acc[mt][n], 0, 0, 0);
                }
            }
        }
    };
    Words w0, w1;
    fetch(0, w0);
    for (int c = 0; c < nchunk; c += 2) {
        if (c + 1 < nchunk) fetch(c + 1, w1);
        compute(c, w0);
        if (c + 2 < nchunk) fetch(c + 2, w0);
        if (c + 1 < nchunk) compute(c + 1, w1);
    }
    // scores (times 1/sqrt d) of the live (token, parent) columns and generator
    // rows; the fused epilogue takes them (standardized with STD) in place first
    const bool all_rows = 32 * MT == D;   // else rows from D on are padding
    const float osc = FUSE ? 1.f : P.rsd;
    auto store_scores = [&](int n) {
        const int col = wc * 64 + n * 16 + c16, tt = col >> csh, q = col & (KC - 1);
        if (tt >= nt_tok || q >= KP) return;
        float* dst = scores + ((tb + tt) * KP + q) * D + wr * 16 * MT + 4 * kq;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            if (all_rows || wr * 16 * MT + 16 * mt + 4 * kq < D) {
                const f32x4 v = acc[mt][n];
                *(float4*)(dst + 16 * mt) = make_float4(v[0] * osc, v[1] * osc, v[2] * osc, v[3] * osc);
            }
        }
    };
    if constexpr (!FUSE) {
#pragma unroll
        for (int n = 0; n < 4; ++n) store_scores(n);
    } else {
        const int K = P.active[l], x32 = (lane ^ 32) << 2;
        const int tpw = 64 >> csh;   // tokens in a wave's 64 columns: 4, 2 or 1
        int32_t pid[4];
#pragma unroll
        for (int n = 0; n < 4; ++n) pid[n] = s_pidx[bcol[n]];
        __syncthreads();   // the staging LDS is free from here on
        // s = acc / sqrt d in place; with standardization z = (s - mu) r, the
        // statistics of child p XOR g_row gathered at an index that is always a
        // feature (generator of a clamped row, parent 0 for padding columns)
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int n = 0; n < 4; ++n)
#pragma unroll
                for (int i = 0; i < 4; ++i) acc[mt][n][i] *= P.rsd;
        if constexpr (STD) {
            const uint32_t* gl = P.gens + P.gens_off[l];
            uint32_t gv[MT][4];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int i = 0; i < 4; ++i) gv[mt][i] = gl[min(wr * 16 * MT + 16 * mt + 4 * kq + i, D - 1)];
            constexpr int MH = MT > 1 ? MT / 2 : 1;   // row tiles per batch of gathers
#pragma unroll
            for (int n = 0; n < 4; ++n) {
                const uint32_t pu = pid[n] >= 0 ? (uint32_t)pid[n] : 0u;
#pragma unroll
                for (int m0 = 0; m0 < MT; m0 += MH) {
                    float2 st[MH][4];
#pragma unroll
                    for (int mt = 0; mt < MH; ++mt)
#pragma unroll
                        for (int i = 0; i < 4; ++i) st[mt][i] = stats[pu ^ gv[m0 + mt][i]];
#pragma unroll
                    for (int mt = 0; mt < MH; ++mt)
#pragma unroll
                        for (int i = 0; i < 4; ++i)
                            acc[m0 + mt][n][i] = (acc[m0 + mt][n][i] - st[mt][i].x) * st[mt][i].y;
                }
            }
        }
        uint32_t* s_top = (uint32_t*)smem;             // [TT][2 row halves][64 lanes]
        uint32_t* s_tau = s_top + TT * 128;           // [TT]
        int* s_cnt = (int*)(s_tau + TT);              // [TT]
        // magnitude key of value i of tile (mt, n): |z| bits + 1, 0 for padding
        auto mk = [&](int mt, int n, int i) -> uint32_t {
            const bool ok = (pid[n] >= 0) & (all_rows | (wr * 16 * MT + 16 * mt + 4 * kq + i < D));
            const uint32_t m = (__float_as_uint(acc[mt][n][i]) & 0x7FFFFFFFu) + 1u;
            return ok ? m : 0u;
        };
        // each lane's largest key per token of this wave
        for (int u = 0; u < tpw; ++u) {
            uint32_t top = 0u;
#pragma unroll
            for (int n = 0; n < 4; ++n) {
                if (((n * 16) >> csh) != u) continue;
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) top = max(top, mk(mt, n, i));
            }
            const int tt = ((wc * 64) >> csh) + u;
            s_top[(tt * 2 + wr) * 64 + lane] = top;
        }
        if ((int)threadIdx.x < TT) s_cnt[threadIdx.x] = 0;
        __syncthreads();
        // tau of each token: the K-th largest distinct key among its 128 lane maxima
        for (int tt = wave; tt < TT; tt += 4) {
            uint32_t v[2];
#pragma unroll
            for (int r = 0; r < 2; ++r) v[r] = s_top[tt * 128 + lane * 2 + r];
            sort_desc<2, 6, false>(v, lane, x32);
            uint32_t prev = (uint32_t)__shfl((int)v[1], (lane + 63) & 63, 64);
            if (lane == 0) prev = 0u;
            int kept = 0, cnt = 0;
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                const bool kk = v[r] != 0u && v[r] != prev;
                kept |= (int)kk << r;
                cnt += (int)kk;
                prev = v[r];
            }
            int total = 0;
            int rank = wave_prefix5(cnt, lane, total);
            uint32_t tau_l = 0u;
#pragma unroll
            for (int r = 0; r < 2; ++r) {
                if (((kept >> r) & 1) && rank == K - 1) tau_l = v[r];
                rank += (kept >> r) & 1;
            }
            const uint64_t hb = __ballot(tau_l != 0u);
            const uint32_t tau = hb ? (uint32_t)__shfl((int)tau_l, __builtin_ctzll(hb), 64) : 1u;
            if (lane == 0) s_tau[tt] = tau;
        }
        __syncthreads();
        // list the candidates at or above tau in the token's region: each
        // lane counts its hits of a column tile, a wave prefix gives its
        // offsets, one LDS atomic per wave and tile reserves the space; the
        // tile's z values go through the wave's LDS rows so that each lane
        // visits only its hits
        float* zrow = (float*)(smem + kWideEpiZ) + (wave * 64 + lane) * (4 * MT + 4);
#pragma unroll
        for (int n = 0; n < 4; ++n) {
            const int tt = bcol[n] >> csh, q = bcol[n] & (KC - 1);
            const uint32_t tau = s_tau[tt];
            uint64_t* lst = (uint64_t*)(scores + (tb + tt) * KP * D);
            uint32_t hm = 0u;   // bit 4 mt + i: value (mt, i) is listed
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int i = 0; i < 4; ++i) hm |= (uint32_t)(mk(mt, n, i) >= tau) << (4 * mt + i);
            int total = 0;
            int pos = wave_prefix<6>(__popc(hm), lane, total);   // at most 4 MT = 32 hits
            int base = 0;
            if (lane == 0 && total > 0) base = atomicAdd(&s_cnt[tt], total);
            pos += __shfl(base, 0, 64);
            if (total == 0) continue;
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const f32x4 v = acc[mt][n];
                *(float4*)(zrow + 4 * mt) = make_float4(v[0], v[1], v[2], v[3]);
            }
            const uint32_t f0 = (uint32_t)(q * D + wr * 16 * MT + 4 * kq);
            while (hm) {
                const int b = __builtin_ctz(hm);
                hm &= hm - 1;
                const uint32_t f = f0 + 16u * (uint32_t)(b >> 2) + (uint32_t)(b & 3);
                if (pos < kWideList) lst[pos] = ((uint64_t)f << 32) | __float_as_uint(zrow[b]);
                ++pos;
            }
        }
        __syncthreads();
        // a token with too many entries gets its full scores instead
#pragma unroll
        for (int n = 0; n < 4; ++n)
            if (s_cnt[bcol[n] >> csh] > kWideList) store_scores(n);
        if ((int)threadIdx.x < nt_tok) counts[tb + threadIdx.x] = s_cnt[threadIdx.x];
    }
}

// Sorts the n <= 64 R keys of the list (0-padded) and emits the first K
// distinct ones of the token into slots [sb, sb + K); returns how many.
template <int R>
__device__ __forceinline__ int wide_emit(const DevPlan& P, const uint64_t* lst, int n, int K, int lane, int x32,
                                         int64_t t, int sb, int32_t* out_idx, float* out_coef)
{
    uint64_t v[R];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const int e = lane * R + r;
        v[r] = e < n ? lst[e] : 0ull;
    }
    sort_desc<R, 6, false>(v, lane, x32);
    uint64_t prev = shfl_u64(v[R - 1], (lane + 63) & 63);
    if (lane == 0) prev = 0ull;
    int kept = 0, cnt = 0;
#pragma unroll
    for (int r = 0; r < R; ++r) {
        const bool k = v[r] != 0ull && v[r] != prev;
        kept |= (int)k << r;
        cnt += (int)k;
        prev = v[r];
    }
    int total = 0;
    int rank = wave_prefix5(cnt, lane, total);
#pragma unroll
    for (int r = 0; r < R; ++r) {
        if (((kept >> r) & 1) && rank < K) {
            out_idx[t * P.k_tot + sb + rank] = (int32_t)key_index(v[r]);
            out_coef[t * P.k_tot + sb + rank] = key_value(v[r]);
        }
        rank += (kept >> r) & 1;
    }
    return total;
}

// counts (plain scores only): the GEMM listed counts[t - t0] <= kWideList
// (candidate, z) entries at or above the threshold in the token's region; more
// means the region holds the full scores.  Without counts the region always
// holds the full scores.
template <bool STD>
__global__ __launch_bounds__(kWideThreads) void wide_select_kernel(DevPlan P, int l, int64_t t0, int64_t ntok,
                                                                   const float* __restrict__ scores,
                                                                   const int* __restrict__ counts,
                                                                   const float2* __restrict__ stats,
                                                                   int32_t* __restrict__ out_idx,
                                                                   float* __restrict__ out_coef)
{
    __shared__ uint64_t s_list[4][64 * kSegStride];
    __shared__ int32_t s_par[4][128];
    __shared__ uint32_t s_gen[256];
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63, x32 = (lane ^ 32) << 2;
    const int KP = P.active[l - 1], D = P.delta[l], K = P.active[l], n = KP * D, sb = P.slot_base[l];
    const int dsh = 31 - __builtin_clz((unsigned)D);
    for (int j = threadIdx.x; j < D; j += kWideThreads) s_gen[j] = P.gens[P.gens_off[l] + j];
    __syncthreads();
    // chunk-relative token (wave-uniform: scalar, so score addresses are 32-bit offsets)
    const int64_t tl = __builtin_amdgcn_readfirstlane((int)blockIdx.x * 4 + wave);
    if (tl >= ntok) return;
    const int64_t t = t0 + tl;
    for (int q = lane; q < KP; q += 64) s_par[wave][q] = out_idx[t * P.k_tot + P.slot_base[l - 1] + q];
    wave_sync();
    // live parent slots as a bit set (padding parents have no children)
    uint64_t live[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int q = 64 * h + lane;
        live[h] = __ballot(q < KP && s_par[wave][q] >= 0);
    }
    const float* src = scores + tl * (int64_t)n;

    // candidate f is child s_gen[f mod D] of parent slot f / D
    auto child_index = [&](int f) -> uint32_t { return (uint32_t)s_par[wave][f >> dsh] ^ s_gen[f & (D - 1)]; };
    auto is_live = [&](int f) -> bool {
        const int q = f >> dsh;
        const uint64_t lw = q < 64 ? live[0] : live[1];
        return f < n && ((lw >> (q & 63)) & 1ull);
    };
    // standardized score of a live candidate
    auto z_of = [&](int f, float v) -> float {
        if constexpr (STD) {
            const float2 st = stats[child_index(f)];
            v = (v - st.x) * st.y;
        }
        return v;
    };
    // magnitude key |z| bits + 1, 0 for padding: distinct values mean distinct children
    auto mkey = [](bool ok, float z) -> uint32_t { return ok ? (__float_as_uint(z) & 0x7FFFFFFFu) + 1u : 0u; };
    // this lane's candidates are streamed from the workspace eight at a time
    // (unconditional, clamped loads: one wait per round)
    constexpr int B = 8;
    const int rounds = (n + 64 * B - 1) / (64 * B);
    auto load_round = [&](int rd, float (&v)[B]) {
#pragma unroll
        for (int b = 0; b < B; ++b)
            v[b] = *(const float*)((const char*)src + 4u * (uint32_t)min((rd * B + b) * 64 + lane, n - 1));
    };

    uint64_t* lst = s_list[wave];
    int nl = kWideList + 1;
    const int listed = counts ? counts[tl] : kWideList + 1;
    if (listed <= kWideList) {
        // the GEMM's list: full keys of its entries
        const uint64_t* ent = (const uint64_t*)src;
        for (int e = lane; e < listed; e += 64) {
            const uint64_t en = ent[e];
            lst[e] = make_key(__uint_as_float((uint32_t)en), child_index((int)(en >> 32)));
        }
        wave_sync();
        nl = listed;
    } else {
        // threshold tau: the K-th largest distinct magnitude key among the lanes'
        // top two.  At least K distinct children have mkey >= tau, so the top K
        // distinct (|z|, index) keys are all among the candidates with mkey >= tau.
        uint32_t top0 = 0u, top1 = 0u;
        for (int rd = 0; rd < rounds; ++rd) {
            float v[B];
            load_round(rd, v);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int f = (rd * B + b) * 64 + lane;
                const bool ok = is_live(f);
                const uint32_t m = mkey(ok, ok ? z_of(f, v[b]) : 0.f);
                const bool gt0 = m > top0, gt1 = m > top1 && m != top0;
                top1 = gt0 ? top0 : (gt1 ? m : top1);
                top0 = gt0 ? m : top0;
            }
        }
        constexpr int M = 2;
        uint32_t top[M] = {top0, top1};
        sort_desc<M, 6, false>(top, lane, x32);
        uint32_t prev = (uint32_t)__shfl((int)top[M - 1], (lane + 63) & 63, 64);
        if (lane == 0) prev = 0u;
        int kept = 0, cnt = 0;
#pragma unroll
        for (int r = 0; r < M; ++r) {
            const bool kk = top[r] != 0u && top[r] != prev;
            kept |= (int)kk << r;
            cnt += (int)kk;
            prev = top[r];
        }
        int total = 0;
        int rank = wave_prefix5(cnt, lane, total);
        uint32_t tau_l = 0u;
#pragma unroll
        for (int r = 0; r < M; ++r) {
            if (((kept >> r) & 1) && rank == K - 1) tau_l = top[r];
            rank += (kept >> r) & 1;
        }
        // one lane holds tau when at least K distinct magnitudes were seen; else take every live candidate
        uint32_t tau = 1u;
        const uint64_t hb = __ballot(tau_l != 0u);
        if (hb) tau = (uint32_t)__shfl((int)tau_l, __builtin_ctzll(hb), 64);

        // collect (f, z) of the candidates with mkey >= tau: each lane appends to
        // its own segment of kSeg entries (every candidate is stored, at the
        // lane's next free entry, so the pass has no branches and no cross-lane
        // steps; entry kSeg takes what does not fit).  The segments are then
        // packed into one list of full keys.  A lane with more than kSeg hits
        // sends the token to the exact extraction below.
        int mine_n = 0;
        for (int rd = 0; rd < rounds; ++rd) {
            float v[B];
            load_round(rd, v);
#pragma unroll
            for (int b = 0; b < B; ++b) {
                const int f = (rd * B + b) * 64 + lane;
                const bool ok = is_live(f);
                const float z = ok ? z_of(f, v[b]) : 0.f;
                lst[lane * kSegStride + min(mine_n, kSeg)] = ((uint64_t)(uint32_t)f << 32) | __float_as_uint(z);
                mine_n += (int)(mkey(ok, z) >= tau);
            }
        }
        wave_sync();
        if (!__ballot(mine_n > kSeg)) {
            uint64_t mine[kSeg];
#pragma unroll
            for (int j = 0; j < kSeg; ++j) {
                mine[j] = 0ull;
                if (j < mine_n) {
                    const uint64_t en = lst[lane * kSegStride + j];
                    mine[j] = make_key(__uint_as_float((uint32_t)en), child_index((int)(en >> 32)));
                }
            }
            const int pre = wave_prefix5(mine_n, lane, nl);
            wave_sync();
#pragma unroll
            for (int j = 0; j < kSeg; ++j)
                if (j < mine_n) lst[pre + j] = mine[j];
        }
        wave_sync();
    }
    int emitted;
    if (nl <= 64) emitted = wide_emit<1>(P, lst, nl, K, lane, x32, t, sb, out_idx, out_coef);
    else if (nl <= 128) emitted = wide_emit<2>(P, lst, nl, K, lane, x32, t, sb, out_idx, out_coef);
    else if (nl <= 256) emitted = wide_emit<4>(P, lst, nl, K, lane, x32, t, sb, out_idx, out_coef);
    else if (nl <= 512) emitted = wide_emit<8>(P, lst, nl, K, lane, x32, t, sb, out_idx, out_coef);
    else if (nl <= kWideList) emitted = wide_emit<16>(P, lst, nl, K, lane, x32, t, sb, out_idx, out_coef);
    else {
        // exact extraction: K rounds of the largest key below the previous one
        uint64_t last = ~0ull;
        emitted = 0;
        for (int r = 0; r < K; ++r) {
            uint64_t best = 0ull;
            for (int rd = 0; rd < rounds; ++rd) {
                float v[B];
                load_round(rd, v);
#pragma unroll
                for (int b = 0; b < B; ++b) {
                    const int f = (rd * B + b) * 64 + lane;
                    const bool ok = is_live(f);
                    const uint64_t k = ok ? make_key(z_of(f, v[b]), child_index(f)) : 0ull;
                    best = (k < last && k > best) ? k : best;
                }
            }
#pragma unroll
            for (int off = 32; off > 0; off >>= 1) {
                const uint64_t o = shfl_u64(best, lane ^ off);
                best = o > best ? o : best;
            }
            if (best == 0ull) break;
            if (lane == 0) {
                out_idx[t * P.k_tot + sb + r] = (int32_t)key_index(best);
                out_coef[t * P.k_tot + sb + r] = key_value(best);
            }
            last = best;
            ++emitted;
        }
    }
    for (int r = emitted + lane; r < K; r += 64) {
        out_idx[t * P.k_tot + sb + r] = -1;
        out_coef[t * P.k_tot + sb + r] = 0.f;
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
    const size_t lds = enc_shared_bytes(P, stats != nullptr) + (size_t)kEncWaves * enc_layout(P, x_bf16, stats != nullptr).bytes;
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

// Tokens per pass of the wide encoder (bounds its workspace).
constexpr int64_t kWideChunkTokens = 16384;

static int wide_max_cands(const DevPlan& P)
{
    int m = 0;
    for (int l = 1; l < P.levels; ++l) m = std::max(m, P.active[l - 1] * P.delta[l]);
    return m;
}

static unsigned wide_level0_lds(const DevPlan& P, bool x_bf16, bool std)
{
    const int ND = (P.dp / 2 + 63) / 64;
    const int listn = P.active[0] * (x_bf16 ? 2 * ND : (P.d + 63) / 64);
    const unsigned per_wave = align16u(x_bf16 ? P.prow * 4 : P.dp * 4) + align16u(listn * 8) +
                              align16u((P.active[0] + 1) * 4) + 16;
    return (std ? align16u(P.d * 8) : 0u) + 4 * per_wave;
}

bool encode_wide_supported(const DevPlan& P, bool x_bf16)
{
    if (P.levels < 2 || P.active[0] > 64 || P.d > 4096) return false;
    if (wide_level0_lds(P, x_bf16, true) > (unsigned)kLdsBudget) return false;
    for (int l = 1; l < P.levels; ++l) {
        const int D = P.delta[l];
        if (D < 16 || D > 256 || (D & (D - 1)) || P.cpt[l] > 128 || P.active[l] > 128) return false;
        if (P.active[l - 1] * D > 64 * 128) return false;
        if (wide_gemm_lds(P, l, x_bf16) > (unsigned)kLdsBudget) return false;
    }
    return true;
}

// Workspace: per chunk token, the scores (or the GEMM's list) of its
// candidates, then one count per chunk token.
static size_t wide_scores_bytes(const DevPlan& P, int64_t ch)
{
    return ((size_t)ch * wide_max_cands(P) * 4 + 255) & ~(size_t)255;
}

static size_t wide_chunk_bytes(const DevPlan& P, int64_t ch)
{
    return ch > 0 ? wide_scores_bytes(P, ch) + (((size_t)ch * 4 + 255) & ~(size_t)255) : 0;
}

size_t encode_wide_workspace_bytes(const DevPlan& P, int64_t T)
{
    return wide_chunk_bytes(P, std::min<int64_t>(T, kWideChunkTokens));
}

// counts != nullptr: the fused epilogue (lists instead of scores); STD: it
// standardizes the scores with `st`.
template <bool XB, bool FUSE, bool STD>
static void launch_wide_gemm(const DevPlan& P, int l, const void* x, int64_t c0, int64_t nc, const int32_t* idx,
                             const float2* st, float* scores, int* counts, hipStream_t stream)
{
    const int TT = kWideCols / P.cpt[l];
    const dim3 grid((unsigned)((nc + TT - 1) / TT));
    const size_t lds = wide_gemm_lds(P, l, XB);
    const int MT = std::max(32, P.delta[l]) / 32;
#define DPB_WG(M)                                                                                             \
    do {                                                                                                      \
        allow_lds(wide_gemm_kernel<XB, M, FUSE, STD>, lds);                                                   \
        hipLaunchKernelGGL((wide_gemm_kernel<XB, M, FUSE, STD>), grid, dim3(kWideThreads), lds, stream, P, l, x, c0, \
                           nc, idx, st, scores, counts);                                                      \
    } while (0)
    if (MT == 1) DPB_WG(1);
    else if (MT == 2) DPB_WG(2);
    else if (MT == 4) DPB_WG(4);
    else DPB_WG(8);
#undef DPB_WG
}

template <bool STD>
static void launch_wide_select(const DevPlan& P, int l, int64_t c0, int64_t nc, const float* scores,
                               const int* counts, const float2* st, int32_t* idx, float* coef, hipStream_t stream)
{
    const dim3 grid((unsigned)((nc + 3) / 4));
    hipLaunchKernelGGL((wide_select_kernel<STD>), grid, dim3(kWideThreads), 0, stream, P, l, c0, nc, scores, counts,
                       st, idx, coef);
}

hipError_t launch_encode_wide(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const float* stats,
                              int32_t* idx, float* coef, void* ws, hipStream_t stream, int64_t chunk)
{
    const float2* st = (const float2*)stats;
    {
        int cus = 256, dev = 0;
        hipDeviceProp_t prop;
        if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
            cus = prop.multiProcessorCount;
        const dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>((T + 3) / 4, (int64_t)cus * 8)));
        const size_t lds = wide_level0_lds(P, x_bf16, st != nullptr);
#define DPB_W0(XB, SD)                                                                                        \
    do {                                                                                                      \
        allow_lds(wide_level0_kernel<XB, SD>, lds);                                                           \
        hipLaunchKernelGGL((wide_level0_kernel<XB, SD>), grid, dim3(kWideThreads), lds, stream, P, x, T, st, idx, \
                           coef);                                                                             \
    } while (0)
        if (x_bf16 && st) DPB_W0(true, true);
        else if (x_bf16) DPB_W0(true, false);
        else if (st) DPB_W0(false, true);
        else DPB_W0(false, false);
#undef DPB_W0
    }
    float* scores = (float*)ws;
    if (chunk <= 0) chunk = kWideChunkTokens;
    int* counts = (int*)((char*)ws + wide_scores_bytes(P, std::min<int64_t>(T, chunk)));
    for (int64_t c0 = 0; c0 < T; c0 += chunk) {
        const int64_t nc = std::min<int64_t>(chunk, T - c0);
        for (int l = 1; l < P.levels; ++l) {
            // the fused epilogue standardizes in place (its lists and scores hold z);
            // otherwise the selection standardizes the full scores
            const bool fuse = wide_fused(P, l);
            if (fuse) {
                if (x_bf16 && st) launch_wide_gemm<true, true, true>(P, l, x, c0, nc, idx, st, scores, counts, stream);
                else if (x_bf16) launch_wide_gemm<true, true, false>(P, l, x, c0, nc, idx, st, scores, counts, stream);
                else if (st) launch_wide_gemm<false, true, true>(P, l, x, c0, nc, idx, st, scores, counts, stream);
                else launch_wide_gemm<false, true, false>(P, l, x, c0, nc, idx, st, scores, counts, stream);
                launch_wide_select<false>(P, l, c0, nc, scores, counts, nullptr, idx, coef, stream);
            } else {
                if (x_bf16) launch_wide_gemm<true, false, false>(P, l, x, c0, nc, idx, st, scores, nullptr, stream);
                else launch_wide_gemm<false, false, false>(P, l, x, c0, nc, idx, st, scores, nullptr, stream);
                if (st) launch_wide_select<true>(P, l, c0, nc, scores, nullptr, st, idx, coef, stream);
                else launch_wide_select<false>(P, l, c0, nc, scores, nullptr, st, idx, coef, stream);
            }
        }
    }
    return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Encoder workspace without allocation: the wide encoder's scratch taken from
// a file-scope device array instead of a caller's buffer.  Each device holds
// its own copy; its address is looked up once per device with that device
// current (scratch_setup) and passed to the kernels like a workspace.  Tokens
// go through in passes sized to the array.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxScratchDevices] = {};
}  // namespace

void* scratch_setup(int device)
{
    if (device < 0 || device >= kMaxScratchDevices) return nullptr;
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (!g_scratch[device]) {
        void* ptr = nullptr;
        if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) == hipSuccess) g_scratch[device] = ptr;
        else (void)hipGetLastError();
    }
    return g_scratch[device];
}

int64_t static_chunk_tokens(const DevPlan& P)
{
    // the largest pass (a multiple of 256 tokens, at most the usual chunk) whose workspace fits
    int64_t ch = kWideChunkTokens;
    while (ch >= kStaticMinChunk && wide_chunk_bytes(P, ch) > kStaticScratchBytes) ch -= 256;
    return ch >= kStaticMinChunk ? ch : 0;
}

}  // namespace dpb
