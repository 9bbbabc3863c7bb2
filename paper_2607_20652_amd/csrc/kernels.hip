// HIP kernels for gfx950 (CDNA4): DPB encode, decode and decode-backward.
//
// Sign generation: the sign of feature i at coordinate iota is the parity of
// (M_iota AND i) (App. A.4, packed-parity equation) -- one AND and one
// popcount per entry, computed in registers.
//
// Encode scores the children of the active parents with the matrix cores:
// for level l and a tile of (token, parent) columns,
//     S[j, (t,p)] = sum_iota gamma_j[iota] * (phi~_p (.) x_t)[iota]
// (§2.2 child-scoring equation), with Gamma_l as the 16 x 32 bf16 A
// fragments (exactly +-1) and the sign-flipped activations as B fragments.
// Products of +-1 with bf16 are exact and accumulate in fp32; fp32 inputs
// are split exactly into three bf16 terms.
#include "dpb_internal.hpp"

namespace dpb {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = kBlock / 64;

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

// float -> bf16 bits, round to nearest even.
__device__ __forceinline__ uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

__device__ __forceinline__ uint32_t parity(uint32_t v) { return __popc(v) & 1u; }

// AbsTopK sort key: |s| (as fp32 bits) first, then the smaller index, with
// the sign of s in bit 0 so that the signed coefficient can be rebuilt.
__device__ __forceinline__ uint64_t make_key(float s, uint32_t idx)
{
    const uint32_t u = __float_as_uint(s);
    return ((uint64_t)(u & 0x7FFFFFFFu) << 32) | (uint64_t)(((0x7FFFFFFFu - idx) << 1) | (u >> 31));
}
__device__ __forceinline__ uint32_t key_index(uint64_t key) { return 0x7FFFFFFFu - ((uint32_t)key >> 1); }
__device__ __forceinline__ float key_value(uint64_t key)
{
    return __uint_as_float((uint32_t)(key >> 32) | (((uint32_t)key & 1u) << 31));
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v)
{
    uint32_t hi = (uint32_t)(v >> 32), lo = (uint32_t)v;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t ohi = (uint32_t)__shfl_xor((int)hi, off, 64);
        const uint32_t olo = (uint32_t)__shfl_xor((int)lo, off, 64);
        if (ohi > hi || (ohi == hi && olo > lo)) {
            hi = ohi;
            lo = olo;
        }
    }
    return ((uint64_t)hi << 32) | lo;
}

__device__ __forceinline__ float wave_sum(float v)
{
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

template <bool BF16>
__device__ __forceinline__ float load_act(const void* p, int64_t i)
{
    if constexpr (BF16) return bf16_bits_to_f32(((const uint16_t*)p)[i]);
    else return ((const float*)p)[i];
}

template <bool BF16>
__device__ __forceinline__ void store_act(void* p, int64_t i, float v)
{
    if constexpr (BF16) ((uint16_t*)p)[i] = (uint16_t)f32_to_bf16_rne(v);
    else ((float*)p)[i] = v;
}

// ---------------------------------------------------------------------------
// Decode: y = sum_s coef_s phi_{idx_s}.  A workgroup takes kCodeTokens tokens;
// each thread owns coordinates iota and walks the token's slots (uniform
// across the workgroup).  Basis slots add coef at their own coordinate;
// hashed slots add +-coef everywhere and are scaled by 1/sqrt(d) once.
// ---------------------------------------------------------------------------
constexpr int kCodeTokens = 8;

template <bool OUT_BF16>
__global__ __launch_bounds__(kBlock) void decode_kernel(DevPlan P, const int32_t* __restrict__ idx,
                                                        const float* __restrict__ coef, int64_t T,
                                                        void* __restrict__ y)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int k = P.k_tot;
    int32_t* s_idx = (int32_t*)smem;
    float* s_coef = (float*)(s_idx + kCodeTokens * k);
    const int64_t t0 = (int64_t)blockIdx.x * kCodeTokens;
    const int ntok = (int)min((int64_t)kCodeTokens, T - t0);
    for (int i = threadIdx.x; i < ntok * k; i += kBlock) {
        s_idx[i] = idx[t0 * k + i];
        s_coef[i] = coef[t0 * k + i];
    }
    __syncthreads();
    for (int tt = 0; tt < ntok; ++tt) {
        const int32_t* ti = s_idx + tt * k;
        const float* tc = s_coef + tt * k;
        for (int iota = threadIdx.x; iota < P.d; iota += kBlock) {
            const uint32_t m = P.masks[iota];
            float acc_b = 0.f, acc_h = 0.f;
            for (int s = 0; s < k; ++s) {
                const int i = ti[s];
                const float a = tc[s];
                if (i < 0) continue;
                if (i < P.d) {
                    if (i == iota) acc_b += a;
                } else {
                    acc_h += __uint_as_float(__float_as_uint(a) ^ (parity(m & (uint32_t)i) << 31));
                }
            }
            store_act<OUT_BF16>(y, (t0 + tt) * P.d + iota, acc_b + P.rsd * acc_h);
        }
    }
}

// ---------------------------------------------------------------------------
// Decode backward: grad_coef[s] = <phi_{idx_s}, g>, then grad_x = decode of
// grad_coef.  One wave reduces one token's slot over the coordinates.
// ---------------------------------------------------------------------------
template <bool G_BF16, bool GX_BF16>
__global__ __launch_bounds__(kBlock) void decode_bwd_kernel(DevPlan P, const int32_t* __restrict__ idx,
                                                            const void* __restrict__ g, int64_t T,
                                                            float* __restrict__ grad_coef,
                                                            void* __restrict__ grad_x, int tpb)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int k = P.k_tot, d = P.d;
    int32_t* s_idx = (int32_t*)smem;            // [tpb][k]
    float* s_gc = (float*)(s_idx + tpb * k);    // [tpb][k]
    float* s_g = s_gc + tpb * k;                // [tpb][d]
    uint32_t* s_m = (uint32_t*)(s_g + tpb * d); // [d]
    const int64_t t0 = (int64_t)blockIdx.x * tpb;
    const int ntok = (int)min((int64_t)tpb, T - t0);
    for (int i = threadIdx.x; i < ntok * k; i += kBlock) s_idx[i] = idx[t0 * k + i];
    for (int i = threadIdx.x; i < ntok * d; i += kBlock) s_g[i] = load_act<G_BF16>(g, t0 * d + i);
    for (int i = threadIdx.x; i < d; i += kBlock) s_m[i] = P.masks[i];
    __syncthreads();

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    for (int tt = wave; tt < ntok; tt += kWaves) {
        const float* gt = s_g + tt * d;
        for (int s = 0; s < k; ++s) {
            const int i = s_idx[tt * k + s];
            float part = 0.f;
            if (i >= d) {
                for (int iota = lane; iota < d; iota += 64)
                    part += __uint_as_float(__float_as_uint(gt[iota]) ^ (parity(s_m[iota] & (uint32_t)i) << 31));
            }
            const float sum = wave_sum(part);
            if (lane == 0) s_gc[tt * k + s] = i < 0 ? 0.f : (i < d ? gt[i] : P.rsd * sum);
        }
    }
    __syncthreads();
    for (int i = threadIdx.x; i < ntok * k; i += kBlock) grad_coef[t0 * k + i] = s_gc[i];
    for (int tt = 0; tt < ntok; ++tt) {
        const int32_t* ti = s_idx + tt * k;
        const float* tc = s_gc + tt * k;
        for (int iota = threadIdx.x; iota < d; iota += kBlock) {
            const uint32_t m = s_m[iota];
            float acc_b = 0.f, acc_h = 0.f;
            for (int s = 0; s < k; ++s) {
                const int i = ti[s];
                const float a = tc[s];
                if (i < 0) continue;
                if (i < d) {
                    if (i == iota) acc_b += a;
                } else {
                    acc_h += __uint_as_float(__float_as_uint(a) ^ (parity(m & (uint32_t)i) << 31));
                }
            }
            store_act<GX_BF16>(grad_x, (t0 + tt) * d + iota, acc_b + P.rsd * acc_h);
        }
    }
}

// ---------------------------------------------------------------------------
// Encode.  A workgroup owns a tile of tokens held in LDS; levels run in turn.
// ---------------------------------------------------------------------------

// B fragment of one (token, parent) column: 8 consecutive coordinates
// starting at `base`, each sign-flipped by parity(M_iota AND p).
__device__ __forceinline__ uint32_t flip_bits8(const uint32_t* s_mask, int base, uint32_t p)
{
    const u32x4 m0 = *(const u32x4*)(s_mask + base);
    const u32x4 m1 = *(const u32x4*)(s_mask + base + 4);
    return parity(m0.x & p) | (parity(m0.y & p) << 1) | (parity(m0.z & p) << 2) | (parity(m0.w & p) << 3) |
           (parity(m1.x & p) << 4) | (parity(m1.y & p) << 5) | (parity(m1.z & p) << 6) | (parity(m1.w & p) << 7);
}

template <bool X_BF16>
__global__ __launch_bounds__(kBlock) void encode_kernel(DevPlan P, const void* __restrict__ xin, int64_t T,
                                                        int32_t* __restrict__ out_idx,
                                                        float* __restrict__ out_coef, int tile_tokens)
{
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int XB = X_BF16 ? 2 : 4;
    const EncodeLayout L = encode_layout(P, XB, tile_tokens);
    const int TT = tile_tokens, d = P.d, dp = P.dp, kmax = P.kmax, k_tot = P.k_tot, cpm = L.cpad_max;
    uint32_t* s_mask = (uint32_t*)smem;
    unsigned char* s_x = smem + L.off_x;
    int32_t* s_par = (int32_t*)(smem + L.off_par);
    uint64_t* s_key = (uint64_t*)(smem + L.off_key);

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int64_t t0 = (int64_t)blockIdx.x * TT;
    const int ntok = (int)min((int64_t)TT, T - t0);

    for (int i = tid; i < dp; i += kBlock) s_mask[i] = P.masks[i];
    for (int i = tid; i < TT * dp; i += kBlock) {
        const int tt = i / dp, iota = i - tt * dp;
        const bool live = tt < ntok && iota < d;
        if constexpr (X_BF16)
            ((uint16_t*)s_x)[i] = live ? ((const uint16_t*)xin)[(t0 + tt) * d + iota] : (uint16_t)0;
        else
            ((float*)s_x)[i] = live ? ((const float*)xin)[(t0 + tt) * d + iota] : 0.f;
    }
    __syncthreads();

    // ---- level 0: AbsTopK over the coordinates (§2.1 Eq. 2: a coordinate read)
    {
        const int K0 = P.active[0];
        const int U = (d + 63) / 64;
        for (int tt = wave; tt < TT; tt += kWaves) {
            if (tt >= ntok) {
                for (int r = lane; r < K0; r += 64) s_par[tt * kmax + r] = -1;
                continue;
            }
            uint64_t taken = 0;
            for (int r = 0; r < K0; ++r) {
                uint64_t best = 0;
                for (int u = 0; u < U; ++u) {
                    const int iota = lane + 64 * u;
                    if (iota >= d || ((taken >> u) & 1u)) continue;
                    float v;
                    if constexpr (X_BF16) v = bf16_bits_to_f32(((const uint16_t*)s_x)[tt * dp + iota]);
                    else v = ((const float*)s_x)[tt * dp + iota];
                    const uint64_t key = make_key(v, (uint32_t)iota);
                    best = key > best ? key : best;
                }
                const uint64_t top = wave_max_u64(best);
                const uint32_t iota = key_index(top);
                if ((int)(iota & 63u) == lane) taken |= (uint64_t)1 << (iota >> 6);
                if (lane == 0) {
                    out_idx[(t0 + tt) * k_tot + r] = (int32_t)iota;
                    out_coef[(t0 + tt) * k_tot + r] = key_value(top);
                    s_par[tt * kmax + r] = (int32_t)iota;
                }
            }
        }
    }

    // ---- levels l >= 1: score the children of the active parents, select
    for (int l = 1; l < P.levels; ++l) {
        __syncthreads();
        const int Kp = P.active[l - 1], Dl = P.delta[l], MB = P.mblocks[l], cp = P.cpad[l];
        const int ncand = Kp * Dl;
        const int ncol = TT * Kp, NB = (ncol + 15) / 16;
        const uint32_t* gens = P.gens + P.gens_off[l];

        for (int i = tid; i < TT * (cp - ncand); i += kBlock) {
            const int tt = i / (cp - ncand);
            s_key[tt * cpm + ncand + (i - tt * (cp - ncand))] = 0;
        }

        const u32x4* gamma = (const u32x4*)P.gamma + P.gamma_off[l];
        for (int item = wave; item < NB * MB; item += kWaves) {
            const int nb = item / MB, mb = item - nb * MB;
            const int col = nb * 16 + (lane & 15);
            const int tt = col / Kp, kk = col - tt * Kp;
            int32_t p = -1;
            if (col < ncol && tt < ntok) p = s_par[tt * kmax + kk];
            const bool cv = p >= 0;
            const uint32_t up = (uint32_t)p;
            const int kq = lane >> 4;
            const int row = cv ? tt : 0;
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
            const u32x4* A = gamma + (int64_t)mb * P.nchunk * 64 + lane;
            for (int c = 0; c < P.nchunk; ++c) {
                const u32x4 a = A[(int64_t)c * 64];
                const int base = c * kChunk + kq * 8;
                const uint32_t sg = cv ? flip_bits8(s_mask, base, up) : 0u;
                if constexpr (X_BF16) {
                    u32x4 b = *(const u32x4*)((const uint16_t*)s_x + row * dp + base);
                    b.x ^= ((sg & 1u) << 15) | (((sg >> 1) & 1u) << 31);
                    b.y ^= (((sg >> 2) & 1u) << 15) | (((sg >> 3) & 1u) << 31);
                    b.z ^= (((sg >> 4) & 1u) << 15) | (((sg >> 5) & 1u) << 31);
                    b.w ^= (((sg >> 6) & 1u) << 15) | (((sg >> 7) & 1u) << 31);
                    if (!cv) b = (u32x4){0u, 0u, 0u, 0u};
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                                   __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
                } else {
                    const float* xr = (const float*)s_x + row * dp + base;
                    uint32_t hi[8], mid[8], lo[8];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        float v = cv ? __uint_as_float(__float_as_uint(xr[e]) ^ (((sg >> e) & 1u) << 31)) : 0.f;
                        hi[e] = f32_to_bf16_rne(v);
                        const float r1 = v - bf16_bits_to_f32(hi[e]);
                        mid[e] = f32_to_bf16_rne(r1);
                        lo[e] = f32_to_bf16_rne(r1 - bf16_bits_to_f32(mid[e]));
                    }
                    const u32x4 bh = {hi[0] | (hi[1] << 16), hi[2] | (hi[3] << 16), hi[4] | (hi[5] << 16),
                                      hi[6] | (hi[7] << 16)};
                    const u32x4 bm = {mid[0] | (mid[1] << 16), mid[2] | (mid[3] << 16), mid[4] | (mid[5] << 16),
                                      mid[6] | (mid[7] << 16)};
                    const u32x4 bl = {lo[0] | (lo[1] << 16), lo[2] | (lo[3] << 16), lo[4] | (lo[5] << 16),
                                      lo[6] | (lo[7] << 16)};
                    const bf16x8 av = __builtin_bit_cast(bf16x8, a);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bh), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bm), acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, __builtin_bit_cast(bf16x8, bl), acc, 0, 0, 0);
                }
            }
            // D fragment: this lane holds rows 4*kq + i of column `col`.
            if (col < ncol) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int j = mb * 16 + kq * 4 + i;
                    if (j < Dl) {
                        const uint64_t key = cv ? make_key(acc[i] * P.rsd, up ^ gens[j]) : 0ull;
                        s_key[tt * cpm + kk * Dl + j] = key;
                    }
                }
            }
        }
        __syncthreads();

        // bitonic sort of each token's cp keys, descending
        for (int size = 2; size <= cp; size <<= 1) {
            for (int stride = size >> 1; stride > 0; stride >>= 1) {
                const int half = cp >> 1;
                for (int e = tid; e < TT * half; e += kBlock) {
                    const int tt = e / half, h = e - tt * half;
                    const int i = 2 * stride * (h / stride) + (h % stride);
                    uint64_t* rowk = s_key + tt * cpm;
                    const uint64_t a = rowk[i], b = rowk[i + stride];
                    const bool desc = (i & size) == 0;
                    if (desc ? (a < b) : (a > b)) {
                        rowk[i] = b;
                        rowk[i + stride] = a;
                    }
                }
                __syncthreads();
            }
        }

        // drop repeated children (adjacent after the sort), keep the first K_l
        const int Kl = P.active[l], sb = P.slot_base[l];
        for (int tt = wave; tt < TT; tt += kWaves) {
            const uint64_t* rowk = s_key + tt * cpm;
            const bool live = tt < ntok;
            int count = 0;
            for (int c0 = 0; c0 < cp && count < Kl; c0 += 64) {
                const int i = c0 + lane;
                const uint64_t key = i < cp ? rowk[i] : 0ull;
                const uint64_t prev = (i > 0 && i < cp) ? rowk[i - 1] : 0ull;
                const bool kept = key != 0ull && !(prev != 0ull && key_index(prev) == key_index(key));
                const uint64_t bal = __ballot(kept);
                const int rank = count + __popcll(bal & ((1ull << lane) - 1ull));
                if (kept && rank < Kl) {
                    const uint32_t ci = key_index(key);
                    s_par[tt * kmax + rank] = (int32_t)ci;
                    if (live) {
                        out_idx[(t0 + tt) * k_tot + sb + rank] = (int32_t)ci;
                        out_coef[(t0 + tt) * k_tot + sb + rank] = key_value(key);
                    }
                }
                count += __popcll(bal);
            }
            for (int r = count + lane; r < Kl; r += 64) {
                s_par[tt * kmax + r] = -1;
                if (live) {
                    out_idx[(t0 + tt) * k_tot + sb + r] = -1;
                    out_coef[(t0 + tt) * k_tot + sb + r] = 0.f;
                }
            }
        }
    }
}

size_t bwd_lds_bytes(const DevPlan& P, int tpb) { return (size_t)tpb * (P.k_tot * 8 + P.d * 4) + (size_t)P.d * 4; }

int bwd_tokens_per_block(const DevPlan& P)
{
    int tpb = kCodeTokens;
    while (tpb > 1 && bwd_lds_bytes(P, tpb) > (size_t)kLdsBudget) --tpb;
    return tpb;
}

int pick_tile_tokens(const DevPlan& P, int x_bytes)
{
    int tt = 16;
    while (tt > 1 && encode_layout(P, x_bytes, tt).bytes > (unsigned)kLdsBudget) --tt;
    return tt;
}

}  // namespace

bool plan_fits(const DevPlan& P)
{
    return encode_layout(P, 4, 1).bytes <= (unsigned)kLdsBudget && bwd_lds_bytes(P, 1) <= (size_t)kLdsBudget &&
           (size_t)kCodeTokens * P.k_tot * 8 <= (size_t)kLdsBudget;
}

hipError_t launch_encode(const DevPlan& P, const void* x, bool x_bf16, int64_t T, int32_t* idx, float* coef,
                         hipStream_t stream)
{
    const int xb = x_bf16 ? 2 : 4;
    const int tt = pick_tile_tokens(P, xb);
    const EncodeLayout L = encode_layout(P, xb, tt);
    if (L.bytes > (unsigned)kLdsBudget) return hipErrorInvalidValue;
    const int64_t blocks = (T + tt - 1) / tt;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    allow_lds(encode_kernel<true>, L.bytes);
    allow_lds(encode_kernel<false>, L.bytes);
    if (x_bf16)
        hipLaunchKernelGGL(encode_kernel<true>, dim3((unsigned)blocks), dim3(kBlock), L.bytes, stream, P, x, T, idx,
                           coef, tt);
    else
        hipLaunchKernelGGL(encode_kernel<false>, dim3((unsigned)blocks), dim3(kBlock), L.bytes, stream, P, x, T,
                           idx, coef, tt);
    return hipGetLastError();
}

hipError_t launch_decode(const DevPlan& P, const int32_t* idx, const float* coef, int64_t T, void* y, bool y_bf16,
                         hipStream_t stream)
{
    const size_t lds = (size_t)kCodeTokens * P.k_tot * 8;
    const int64_t blocks = (T + kCodeTokens - 1) / kCodeTokens;
    if (lds > (size_t)kLdsBudget || blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    if (y_bf16)
        hipLaunchKernelGGL(decode_kernel<true>, dim3((unsigned)blocks), dim3(kBlock), lds, stream, P, idx, coef, T, y);
    else
        hipLaunchKernelGGL(decode_kernel<false>, dim3((unsigned)blocks), dim3(kBlock), lds, stream, P, idx, coef, T, y);
    return hipGetLastError();
}

hipError_t launch_decode_bwd(const DevPlan& P, const int32_t* idx, const void* g, bool g_bf16, int64_t T,
                             float* grad_coef, void* grad_x, bool gx_bf16, hipStream_t stream)
{
    const int tpb = bwd_tokens_per_block(P);
    const size_t lds = bwd_lds_bytes(P, tpb);
    const int64_t blocks = (T + tpb - 1) / tpb;
    if (lds > (size_t)kLdsBudget || blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const dim3 grid((unsigned)blocks), block(kBlock);
    if (g_bf16 && gx_bf16)
        hipLaunchKernelGGL((decode_bwd_kernel<true, true>), grid, block, lds, stream, P, idx, g, T, grad_coef, grad_x, tpb);
    else if (g_bf16)
        hipLaunchKernelGGL((decode_bwd_kernel<true, false>), grid, block, lds, stream, P, idx, g, T, grad_coef, grad_x, tpb);
    else if (gx_bf16)
        hipLaunchKernelGGL((decode_bwd_kernel<false, true>), grid, block, lds, stream, P, idx, g, T, grad_coef, grad_x, tpb);
    else
        hipLaunchKernelGGL((decode_bwd_kernel<false, false>), grid, block, lds, stream, P, idx, g, T, grad_coef, grad_x, tpb);
    return hipGetLastError();
}

}  // namespace dpb
