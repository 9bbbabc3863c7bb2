// Encoder for gfx950: the top-down beam search of §2.2.
//
// A wave owns `wave_tokens` tokens; their activations stay in LDS in the
// paired layout of scoring.hpp.
//
//  * Level 0 (§2.1 Eq. 2: scoring a basis feature is a coordinate read):
//    each token's lanes take the maximum key over their coordinates; the
//    K_0-th largest lane maximum tau bounds the answer from below (the K_0
//    largest lane maxima are distinct keys >= tau), so only keys >= tau --
//    at most K_0 lanes' worth -- are ranked exactly.
//  * Levels l >= 1: the children of every active parent are scored on the
//    matrix cores; the keys (|s| desc, index asc, see device_common.hpp) are
//    sorted in registers by a bitonic network laid over the MFMA output
//    layout; a child reached from several parents has bit-identical keys
//    (same products, same reduction), so it appears as adjacent duplicates
//    and is kept once; the first K_l survivors are emitted in order.
#include <algorithm>

#include "scoring.hpp"

namespace dpb {
namespace {

constexpr int kEncWaves = 4;
constexpr int kEncThreads = 64 * kEncWaves;

struct EncLayout {
    unsigned act, cw, par, list, bytes;
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
    const int U0 = (P.dp + LPT - 1) / LPT;
    const int R = enc_r(P);
    int listn = P.active[0] * U0;
    for (int l = 1; l < P.levels; ++l) listn = P.cpt[l] * 4 * R > listn ? P.cpt[l] * 4 * R : listn;
    L.listn = listn;
    L.kmaxp = P.kmax;
    unsigned off = 0;
    L.act = off;
    off = align16u(off + (act_bf16 ? TPW * (P.dp * 2 + P.nchunk * 4) : TPW * P.dp * 4));
    L.cw = off;   off = align16u(off + 16 * P.cws * 4);
    L.par = off;  off = align16u(off + TPW * L.kmaxp * 4);
    L.list = off; off = align16u(off + TPW * listn * 8);
    L.bytes = off;
    return L;
}

__host__ __device__ inline unsigned enc_shared_bytes(const DevPlan& P)
{
    return align16u(P.dp * 4) + align16u(P.nt_groups * 16 * P.nchunk * 4);
}

__device__ __forceinline__ uint64_t shfl_xor64(uint64_t v, int mask)
{
    const uint32_t hi = (uint32_t)__shfl_xor((int)(v >> 32), mask, 64);
    const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)v, mask, 64);
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ uint64_t shfl64(uint64_t v, int src)
{
    const uint32_t hi = (uint32_t)__shfl((int)(v >> 32), src, 64);
    const uint32_t lo = (uint32_t)__shfl((int)(uint32_t)v, src, 64);
    return ((uint64_t)hi << 32) | lo;
}

// Descending bitonic sort of one token's keys: element e = lanepos * R + r
// lives in register r of the lane whose position is lanepos.  Bits of lanepos
// map to lane bits through `lane_xor(b)`.  nbits = log2(R) + bits of lanepos.
template <int R, typename LaneXor>
__device__ void bitonic_desc(uint64_t (&v)[R], int lanepos, int nbits, LaneXor lane_xor)
{
    constexpr int LR = R == 4 ? 2 : R == 8 ? 3 : R == 16 ? 4 : R == 2 ? 1 : 0;
    for (int ks = 1; ks <= nbits; ++ks) {
        const int k = 1 << ks;
        for (int js = ks - 1; js >= 0; --js) {
            const int j = 1 << js;
            if (js >= LR) {
                const int m = lane_xor(js - LR);
#pragma unroll
                for (int r = 0; r < R; ++r) {
                    const uint64_t o = shfl_xor64(v[r], m);
                    const int e = lanepos * R + r;
                    const bool take_max = ((e & j) == 0) == ((e & k) == 0);
                    v[r] = take_max ? (o > v[r] ? o : v[r]) : (o < v[r] ? o : v[r]);
                }
            } else {
#pragma unroll
                for (int jj = 1; jj < R; jj <<= 1) {
                    if (jj != j) continue;
#pragma unroll
                    for (int r = 0; r < R; ++r) {
                        if (r & jj) continue;
                        const bool desc = ((lanepos * R + r) & k) == 0;
                        const uint64_t a = v[r], b = v[r | jj];
                        const bool sw = desc ? (a < b) : (a > b);
                        v[r] = sw ? b : a;
                        v[r | jj] = sw ? a : b;
                    }
                }
            }
        }
    }
}

// Emits the first K distinct keys of each token's sorted list (duplicates are
// adjacent) to slots [sb, sb + K), and records them as the next parents.
__device__ void emit_level(const DevPlan& P, int lane, int64_t t0, int ntok, const uint64_t* list, int listn, int n,
                           int K, int sb, int32_t* par, int kmaxp, int32_t* out_idx, float* out_coef)
{
    const int TPW = P.wave_tokens, LPT = 64 / TPW, tt = lane / LPT, li = lane % LPT, k_tot = P.k_tot;
    const uint64_t block = LPT == 64 ? ~0ull : (((1ull << LPT) - 1ull) << (tt * LPT));
    const bool live = tt < ntok;
    const uint64_t* row = list + tt * listn;
    int count = 0;
    for (int e0 = 0; e0 < n; e0 += LPT) {
        const int e = e0 + li;
        const uint64_t key = e < n ? row[e] : 0ull;
        const uint64_t prev = (e > 0 && e < n) ? row[e - 1] : 0ull;
        const bool kept = key != 0ull && key != prev;
        const uint64_t m = __ballot(kept) & block;
        const int rank = count + __popcll(m & ((1ull << lane) - 1ull));
        if (kept && rank < K) {
            const uint32_t ci = key_index(key);
            par[tt * kmaxp + rank] = (int32_t)ci;
            if (live) {
                out_idx[(t0 + tt) * k_tot + sb + rank] = (int32_t)ci;
                out_coef[(t0 + tt) * k_tot + sb + rank] = key_value(key);
            }
        }
        count += __popcll(m);
    }
    for (int r = count + li; r < K; r += LPT) {
        par[tt * kmaxp + r] = -1;
        if (live) {
            out_idx[(t0 + tt) * k_tot + sb + r] = -1;
            out_coef[(t0 + tt) * k_tot + sb + r] = 0.f;
        }
    }
}

template <bool X_BF16, int R>
__global__ __launch_bounds__(kEncThreads) void encode2_kernel(DevPlan P, const void* __restrict__ xin, int64_t T,
                                                              int32_t* __restrict__ out_idx,
                                                              float* __restrict__ out_coef)
{
    extern __shared__ __align__(16) unsigned char smem[];
    {
        uint32_t* s_mask = (uint32_t*)smem;
        uint32_t* s_nt = (uint32_t*)(smem + align16u(P.dp * 4));
        for (int i = threadIdx.x; i < P.dp; i += kEncThreads) s_mask[i] = P.masks[i];
        for (int i = threadIdx.x; i < P.nt_groups * 16 * P.nchunk; i += kEncThreads) s_nt[i] = P.nt[i];
    }
    __syncthreads();
    const uint32_t* s_nt = (const uint32_t*)(smem + align16u(P.dp * 4));

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int TPW = P.wave_tokens, LPT = 64 / TPW, d = P.d, dp = P.dp, nchunk = P.nchunk;
    const EncLayout EL = enc_layout(P, X_BF16);
    unsigned char* wb = smem + enc_shared_bytes(P) + (unsigned)wave * EL.bytes;
    uint32_t* pairs = (uint32_t*)(wb + EL.act);
    uint32_t* signw = pairs + TPW * (dp / 2);
    float* xf = (float*)(wb + EL.act);
    uint32_t* cw = (uint32_t*)(wb + EL.cw);
    int32_t* par = (int32_t*)(wb + EL.par);
    uint64_t* list = (uint64_t*)(wb + EL.list);
    const ActTile A{pairs, signw, xf};

    const int64_t ngroups = (T + TPW - 1) / TPW;
    for (int64_t grp = (int64_t)blockIdx.x * kEncWaves + wave; grp < ngroups;
         grp += (int64_t)gridDim.x * kEncWaves) {
        const int64_t t0 = grp * TPW;
        const int ntok = (int)min((int64_t)TPW, T - t0);

        if constexpr (X_BF16) {
            load_pairs(P, lane, ntok, TPW, (const uint16_t*)xin, t0, pairs, signw);
        } else {
            const float* xs = (const float*)xin;
            for (int e = lane; e < TPW * dp; e += 64) {
                const int tt = e / dp, iota = e - tt * dp;
                xf[e] = (tt < ntok && iota < d) ? xs[(t0 + tt) * d + iota] : 0.f;
            }
        }
        wave_sync();

        // ---- level 0
        {
            const int tt = lane / LPT, li = lane % LPT, K0 = P.active[0];
            const int U0 = (dp + LPT - 1) / LPT;
            const bool live = tt < ntok;
            auto key0 = [&](int u) -> uint64_t {
                const int iota = li + LPT * u;
                if (!live || iota >= d) return 0ull;
                float v;
                if constexpr (X_BF16) v = pair_value(P, pairs, signw, tt, iota);
                else v = xf[tt * dp + iota];
                return make_key(v, (uint32_t)iota);
            };
            uint64_t best = 0;
            for (int u = 0; u < U0; ++u) {
                const uint64_t kk = key0(u);
                best = kk > best ? kk : best;
            }
            // the K0-th largest lane maximum of the token
            uint64_t sv[1] = {best};
            int lb = 0;
            while ((1 << lb) < LPT) ++lb;
            bitonic_desc<1>(sv, li, lb, [](int b) { return 1 << b; });
            const uint64_t tau = shfl64(sv[0], tt * LPT + K0 - 1);
            int cnt = 0;
            for (int u = 0; u < U0; ++u) cnt += key0(u) >= tau && tau != 0ull;
            int incl = cnt;
            for (int off = 1; off < LPT; off <<= 1) {
                const int o = __shfl_up(incl, off, LPT);
                if (li >= off) incl += o;
            }
            const int total = __shfl(incl, tt * LPT + LPT - 1, 64);
            int pos = incl - cnt;
            uint64_t* row = list + tt * EL.listn;
            for (int u = 0; u < U0; ++u) {
                const uint64_t kk = key0(u);
                if (kk >= tau && tau != 0ull) row[pos++] = kk;
            }
            wave_sync();
            for (int e = li; e < total; e += LPT) {
                const uint64_t ke = row[e];
                int rank = 0;
                for (int f = 0; f < total; ++f) rank += row[f] > ke;
                if (rank < K0) {
                    const uint32_t iota = key_index(ke);
                    par[tt * EL.kmaxp + rank] = (int32_t)iota;
                    if (live) {
                        out_idx[(t0 + tt) * P.k_tot + rank] = (int32_t)iota;
                        out_coef[(t0 + tt) * P.k_tot + rank] = key_value(ke);
                    }
                }
            }
            for (int r = total + li; r < K0; r += LPT) par[tt * EL.kmaxp + r] = -1;
            wave_sync();
        }

        // ---- levels l >= 1
        for (int l = 1; l < P.levels; ++l) {
            const int CPT = P.cpt[l], Kp = P.active[l - 1], Dl = P.delta[l];
            column_bitmaps<X_BF16>(P, lane, ntok, l, 0, par, EL.kmaxp, Kp, A, s_nt, cw);
            wave_sync();
            const int col = lane & 15, kq = lane >> 4;
            const int tt = col / CPT, q = col % CPT;
            const int32_t p = (col < TPW * CPT && tt < ntok && q < Kp) ? par[tt * EL.kmaxp + q] : -1;
            const bool valid = p >= 0;
            const int trow = valid ? tt : 0;
            const uint32_t* gens = P.gens + P.gens_off[l];
            uint64_t keys[R];
#pragma unroll
            for (int mb = 0; mb < R / 4; ++mb) {
                f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                if (mb < P.mblocks[l]) acc = mfma_scores<X_BF16>(P, lane, l, mb, valid, trow, A, cw);
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = 16 * mb + 4 * kq + i;
                    keys[4 * mb + i] =
                        (valid && j < Dl) ? make_key(acc[i] * P.rsd, (uint32_t)p ^ gens[j]) : 0ull;
                }
            }
            int cb = 0;
            while ((1 << cb) < CPT) ++cb;
            const int lanepos = q * 4 + kq;
            int lr = 0;
            while ((1 << lr) < R) ++lr;
            bitonic_desc<R>(keys, lanepos, lr + 2 + cb, [](int b) { return b < 2 ? (16 << b) : (1 << (b - 2)); });
            if (col < TPW * CPT) {
#pragma unroll
                for (int r = 0; r < R; ++r) list[tt * EL.listn + lanepos * R + r] = keys[r];
            }
            wave_sync();
            emit_level(P, lane, t0, ntok, list, EL.listn, CPT * 4 * R, P.active[l], P.slot_base[l], par, EL.kmaxp,
                       out_idx, out_coef);
            wave_sync();
        }
    }
}

}  // namespace

bool encode2_supported(const DevPlan& P)
{
    const int TPW = P.wave_tokens, LPT = 64 / TPW;
    if (P.active[0] > LPT || enc_r(P) > 16) return false;
    for (int l = 1; l < P.levels; ++l)
        if (P.cpt[l] > 16 || TPW * P.cpt[l] > 16) return false;
    const size_t lds = enc_shared_bytes(P) + (size_t)kEncWaves * enc_layout(P, false).bytes;
    return lds <= (size_t)kLdsBudget;
}

hipError_t launch_encode2(const DevPlan& P, const void* x, bool x_bf16, int64_t T, int32_t* idx, float* coef,
                          hipStream_t stream)
{
    const size_t lds = enc_shared_bytes(P) + (size_t)kEncWaves * enc_layout(P, x_bf16).bytes;
    const int64_t groups = (T + P.wave_tokens - 1) / P.wave_tokens;
    const int64_t need = (groups + kEncWaves - 1) / kEncWaves;
    int cus = 256, dev = 0;
    hipDeviceProp_t prop;
    if (hipGetDevice(&dev) == hipSuccess && hipGetDeviceProperties(&prop, dev) == hipSuccess)
        cus = prop.multiProcessorCount;
    const int per_cu = (int)std::max<size_t>(1, (160 * 1024) / std::max<size_t>(lds, 1));
    const dim3 grid((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, (int64_t)cus * std::min(per_cu, 8) * 4)));
    const int R = enc_r(P);
#define DPB_ENC(XB, RV)                                                                                       \
    do {                                                                                                      \
        allow_lds(encode2_kernel<XB, RV>, lds);                                                               \
        hipLaunchKernelGGL((encode2_kernel<XB, RV>), grid, dim3(kEncThreads), lds, stream, P, x, T, idx, coef); \
    } while (0)
    if (x_bf16) {
        if (R == 4) DPB_ENC(true, 4);
        else if (R == 8) DPB_ENC(true, 8);
        else DPB_ENC(true, 16);
    } else {
        if (R == 4) DPB_ENC(false, 4);
        else if (R == 8) DPB_ENC(false, 8);
        else DPB_ENC(false, 16);
    }
#undef DPB_ENC
    return hipGetLastError();
}

}  // namespace dpb
