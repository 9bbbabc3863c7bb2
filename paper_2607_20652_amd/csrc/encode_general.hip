// General encoder for gfx950: the top-down beam search of §2.2 for plans the
// narrow encoder (encode.hip: every level's candidates in one wave's
// registers) and the wide encoder (many children per parent, with a
// workspace) do not cover -- e.g. full generator sets of thousands of
// children per parent, or more level-0 features than a wave has lanes.
//
// Encode scores the children of the active parents with the matrix cores:
// for level l and a tile of (token, parent) columns,
//     S[j, (t,p)] = sum_iota gamma_j[iota] * (phi~_p (.) x_t)[iota]
// (§2.2 child-scoring equation), with Gamma_l as the 16 x 32 bf16 A
// fragments (exactly +-1) and the sign-flipped activations as B fragments,
// the sign of feature p at coordinate iota being the parity of (M_iota AND p)
// (App. A.4, packed-parity equation).  Products of +-1 with bf16 are exact
// and accumulate in fp32; fp32 inputs are split exactly into three bf16
// terms.  The keys of a token's candidates are sorted in LDS by a bitonic
// network over the workgroup.  With statistics (STD) every score is first
// standardized, z = (s - mu) r with the candidate's (mu, r) (§2.2 "Score
// Standardization"), in the same fp32 arithmetic as the other encoders.
#include "device_common.hpp"

namespace dpb {
namespace {

constexpr int kWaves = kBlock / 64;

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

template <bool X_BF16, bool STD>
__global__ __launch_bounds__(kBlock) void encode_kernel(DevPlan P, const void* __restrict__ xin, int64_t T,
                                                        const float2* __restrict__ stats,
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
                    if constexpr (STD) {
                        const float2 st = stats[iota];
                        v = (v - st.x) * st.y;
                    }
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
                        float sc = acc[i] * P.rsd;
                        if constexpr (STD)
                            if (cv) {
                                const float2 st = stats[up ^ gens[j]];
                                sc = (sc - st.x) * st.y;
                            }
                        const uint64_t key = cv ? make_key(sc, up ^ gens[j]) : 0ull;
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

int pick_tile_tokens(const DevPlan& P, int x_bytes)
{
    int tt = 16;
    while (tt > 1 && encode_layout(P, x_bytes, tt).bytes > (unsigned)kLdsBudget) --tt;
    return tt;
}

}  // namespace

bool general_encoder_fits(const DevPlan& P) { return encode_layout(P, 4, 1).bytes <= (unsigned)kLdsBudget; }

hipError_t launch_encode(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const float* stats, int32_t* idx,
                         float* coef, hipStream_t stream)
{
    const int xb = x_bf16 ? 2 : 4;
    const int tt = pick_tile_tokens(P, xb);
    const EncodeLayout L = encode_layout(P, xb, tt);
    if (L.bytes > (unsigned)kLdsBudget) return hipErrorInvalidValue;
    const int64_t blocks = (T + tt - 1) / tt;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const float2* st = (const float2*)stats;
#define DPB_GEN(XB, SD)                                                                                           \
    do {                                                                                                          \
        allow_lds(encode_kernel<XB, SD>, L.bytes);                                                                \
        hipLaunchKernelGGL((encode_kernel<XB, SD>), dim3((unsigned)blocks), dim3(kBlock), L.bytes, stream, P, x, T, \
                           st, idx, coef, tt);                                                                    \
    } while (0)
    if (x_bf16 && st) DPB_GEN(true, true);
    else if (x_bf16) DPB_GEN(true, false);
    else if (st) DPB_GEN(false, true);
    else DPB_GEN(false, false);
#undef DPB_GEN
    return hipGetLastError();
}

}  // namespace dpb
