// Row epilogues and code utilities around the DPB path, for gfx950:
//
//  * normalized reconstruction (§2.2 "Normalized Reconstruction"): the
//    decoder output u of a token is rescaled to the norm of the bottleneck
//    input ref, y = u ||ref|| / ||u||, and its backward;
//  * code edits of the greedy feature editing of App. C.3 (zero, replace or
//    rescale one slot position of a source code from a target code);
//  * the variance auxiliary loss (§2.2 "Auxillary losses") over the active
//    features of a batch, and its gradient with respect to the coefficients.
//
// The row kernels give each wave one row at a time (grid-stride), 8 elements
// per lane per 16- or 32-byte access, and reduce with wave sums: they are
// bound by HBM traffic.
#include <algorithm>

#include "dpb_internal.hpp"

#include "device_common.hpp"
#include "../../include/dpb.h"

namespace dpb {
namespace {

constexpr int kRowWaves = 4;
constexpr int kRowThreads = 64 * kRowWaves;

// 8 consecutive elements at p + i (bf16 or fp32), zero past n.
__device__ __forceinline__ void load8(const void* p, bool bf16, int64_t i, int64_t n, bool vec, float (&v)[8])
{
    if (vec) {
        if (bf16) {
            const u32x4 q = *(const u32x4*)((const uint16_t*)p + i);
            const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[2 * e] = bf16_bits_to_f32(w[e] & 0xFFFFu);
                v[2 * e + 1] = bf16_bits_to_f32(w[e] >> 16);
            }
        } else {
            const float4 a = *(const float4*)((const float*)p + i), b = *(const float4*)((const float*)p + i + 4);
            v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
            v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            v[e] = (i + e < n) ? (bf16 ? bf16_bits_to_f32(((const uint16_t*)p)[i + e]) : ((const float*)p)[i + e]) : 0.f;
    }
}

__device__ __forceinline__ void store8(void* p, bool bf16, int64_t i, int64_t n, bool vec, const float (&v)[8])
{
    if (vec) {
        if (bf16) {
            u32x4 q;
            q.x = pack_bf16x2(v[0], v[1]);
            q.y = pack_bf16x2(v[2], v[3]);
            q.z = pack_bf16x2(v[4], v[5]);
            q.w = pack_bf16x2(v[6], v[7]);
            *(u32x4*)((uint16_t*)p + i) = q;
        } else {
            *(float4*)((float*)p + i) = make_float4(v[0], v[1], v[2], v[3]);
            *(float4*)((float*)p + i + 4) = make_float4(v[4], v[5], v[6], v[7]);
        }
    } else {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (i + e < n) {
                if (bf16) ((uint16_t*)p)[i + e] = (uint16_t)f32_to_bf16_rne(v[e]);
                else ((float*)p)[i + e] = v[e];
            }
    }
}

struct RowIO {
    const void* a; bool a16;
    const void* b; bool b16;
    const void* c; bool c16;
    void* o1; bool o116;
    void* o2; bool o216;
};

// Row t of a [T, d] tensor as NCH chunks of 512 elements, 8 per lane
// (elements 512c + 8 lane + e); lanes past d hold zeros.  NCH = 0 streams the
// row chunk by chunk instead (any d), reading it twice.
template <int NCH>
__device__ __forceinline__ void load_row(const void* p, bool bf16, int64_t r0, int d, int lane, bool vec,
                                         float (&v)[NCH > 0 ? NCH : 1][8])
{
#pragma unroll
    for (int c = 0; c < (NCH > 0 ? NCH : 1); ++c) {
        const int o = 512 * c + lane * 8;
        if (o < d) load8(p, bf16, r0 + o, r0 + d, vec, v[c]);
        else
#pragma unroll
            for (int e = 0; e < 8; ++e) v[c][e] = 0.f;
    }
}

template <int NCH>
__device__ __forceinline__ void store_row(void* p, bool bf16, int64_t r0, int d, int lane, bool vec,
                                          const float (&v)[NCH > 0 ? NCH : 1][8])
{
#pragma unroll
    for (int c = 0; c < (NCH > 0 ? NCH : 1); ++c) {
        const int o = 512 * c + lane * 8;
        if (o < d) store8(p, bf16, r0 + o, r0 + d, vec, v[c]);
    }
}

// y = u * ||ref|| / ||u|| per row (0 when ||u|| = 0); norms[t] = (||ref||, ||u||).
// Row t's reference is row ref_rows[t] of ref when ref_rows is given (norm 0
// when that index is outside [0, T_ref)).  With NCH > 0 (d <= 512 NCH) the
// rows stay in registers between the reduction and the scaling.
template <int NCH>
__global__ __launch_bounds__(kRowThreads) void normalize_kernel(RowIO io, int d, int64_t T, const int32_t* ref_rows,
                                                                int64_t T_ref, float* norms)
{
    constexpr int NC = NCH > 0 ? NCH : 1;
    const int lane = threadIdx.x & 63;
    const bool vec = (d & 7) == 0;
    for (int64_t t = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6); t < T; t += (int64_t)gridDim.x * kRowWaves) {
        const int64_t r0 = t * d;
        const int64_t rr = ref_rows ? (int64_t)ref_rows[t] : t;
        const bool has_ref = rr >= 0 && rr < T_ref;
        const int64_t q0 = has_ref ? rr * d : 0;
        float su = 0.f, sr = 0.f;
        float u[NC][8], r[NC][8];
        if constexpr (NCH > 0) {
            load_row<NCH>(io.a, io.a16, r0, d, lane, vec, u);
            if (has_ref) load_row<NCH>(io.b, io.b16, q0, d, lane, vec, r);
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    su += u[c][e] * u[c][e];
                    if (has_ref) sr += r[c][e] * r[c][e];
                }
        } else {
            for (int o = lane * 8; o < d; o += 512) {
                load8(io.a, io.a16, r0 + o, r0 + d, vec, u[0]);
#pragma unroll
                for (int e = 0; e < 8; ++e) su += u[0][e] * u[0][e];
                if (has_ref) {
                    load8(io.b, io.b16, q0 + o, q0 + d, vec, r[0]);
#pragma unroll
                    for (int e = 0; e < 8; ++e) sr += r[0][e] * r[0][e];
                }
            }
        }
        su = wave_sum(su);
        sr = wave_sum(sr);
        const float nu = sqrtf(su), nr = sqrtf(sr);
        const float scale = nu > 0.f ? nr / nu : 0.f;
        if constexpr (NCH > 0) {
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) u[c][e] *= scale;
            store_row<NCH>(io.o1, io.o116, r0, d, lane, vec, u);
        } else {
            for (int o = lane * 8; o < d; o += 512) {
                load8(io.a, io.a16, r0 + o, r0 + d, vec, u[0]);
#pragma unroll
                for (int e = 0; e < 8; ++e) u[0][e] *= scale;
                store8(io.o1, io.o116, r0 + o, r0 + d, vec, u[0]);
            }
        }
        if (lane == 0 && norms) {
            norms[2 * t] = nr;
            norms[2 * t + 1] = nu;
        }
    }
}

// grad_u = s (g - (<g,u>/||u||^2) u), grad_ref (+)= (<g,u> / (||u|| ||ref||)) ref.
template <int NCH>
__global__ __launch_bounds__(kRowThreads) void normalize_bwd_kernel(RowIO io, int d, int64_t T, int accumulate)
{
    constexpr int NC = NCH > 0 ? NCH : 1;
    const int lane = threadIdx.x & 63;
    const bool vec = (d & 7) == 0;
    for (int64_t t = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6); t < T; t += (int64_t)gridDim.x * kRowWaves) {
        const int64_t r0 = t * d;
        float su = 0.f, sr = 0.f, gu = 0.f;
        float g[NC][8], u[NC][8], r[NC][8];
        if constexpr (NCH > 0) {
            load_row<NCH>(io.a, io.a16, r0, d, lane, vec, g);
            load_row<NCH>(io.b, io.b16, r0, d, lane, vec, u);
            load_row<NCH>(io.c, io.c16, r0, d, lane, vec, r);
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    su += u[c][e] * u[c][e];
                    sr += r[c][e] * r[c][e];
                    gu += g[c][e] * u[c][e];
                }
        } else {
            for (int o = lane * 8; o < d; o += 512) {
                load8(io.a, io.a16, r0 + o, r0 + d, vec, g[0]);
                load8(io.b, io.b16, r0 + o, r0 + d, vec, u[0]);
                load8(io.c, io.c16, r0 + o, r0 + d, vec, r[0]);
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    su += u[0][e] * u[0][e];
                    sr += r[0][e] * r[0][e];
                    gu += g[0][e] * u[0][e];
                }
            }
        }
        su = wave_sum(su);
        sr = wave_sum(sr);
        gu = wave_sum(gu);
        const float nu = sqrtf(su), nr = sqrtf(sr);
        const float s = nu > 0.f ? nr / nu : 0.f;
        const float cu = nu > 0.f ? s * gu / su : 0.f;
        const float cr = (nu > 0.f && nr > 0.f) ? gu / (nu * nr) : 0.f;
        if constexpr (NCH > 0) {
            float a[NC][8];
            if (accumulate) load_row<NCH>(io.o2, io.o216, r0, d, lane, vec, a);
#pragma unroll
            for (int c = 0; c < NC; ++c)
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    u[c][e] = s * g[c][e] - cu * u[c][e];
                    a[c][e] = (accumulate ? a[c][e] : 0.f) + cr * r[c][e];
                }
            store_row<NCH>(io.o1, io.o116, r0, d, lane, vec, u);
            store_row<NCH>(io.o2, io.o216, r0, d, lane, vec, a);
        } else {
            for (int o = lane * 8; o < d; o += 512) {
                float a[8];
                load8(io.a, io.a16, r0 + o, r0 + d, vec, g[0]);
                load8(io.b, io.b16, r0 + o, r0 + d, vec, u[0]);
                load8(io.c, io.c16, r0 + o, r0 + d, vec, r[0]);
#pragma unroll
                for (int e = 0; e < 8; ++e) u[0][e] = s * g[0][e] - cu * u[0][e];
                store8(io.o1, io.o116, r0 + o, r0 + d, vec, u[0]);
                if (accumulate) load8(io.o2, io.o216, r0 + o, r0 + d, vec, a);
#pragma unroll
                for (int e = 0; e < 8; ++e) a[e] = (accumulate ? a[e] : 0.f) + cr * r[0][e];
                store8(io.o2, io.o216, r0 + o, r0 + d, vec, a);
            }
        }
    }
}

// One thread per output slot (e, s): copies source row rows[e] and applies
// the edit at slot position slots[e].
__global__ void edit_kernel(const int32_t* idx, const float* coef, const int32_t* tidx, const float* tcoef,
                            int64_t T, int k, const int32_t* rows, const int32_t* slots, const int32_t* ops,
                            int64_t E, int32_t* out_idx, float* out_coef)
{
    const int64_t n = E * k;
    for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < n; o += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = o / k;
        const int s = (int)(o - e * k);
        const int64_t r = rows[e];
        const int p = slots[e], op = ops[e];
        const bool has_t = tidx != nullptr;
        const bool ok = r >= 0 && r < T && p >= 0 && p < k &&
                        (op == DPB_EDIT_ZERO || op == DPB_EDIT_NONE ||
                         (has_t && (op == DPB_EDIT_REPLACE || op == DPB_EDIT_RESCALE)));
        int32_t i = -1;
        float c = 0.f;
        if (ok) {
            const int64_t src = r * k + s;
            i = idx[src];
            c = coef[src];
            if (s == p) {
                if (op == DPB_EDIT_ZERO) c = 0.f;
                else if (op == DPB_EDIT_REPLACE) {
                    i = tidx[src];
                    c = tcoef[src];
                } else if (op == DPB_EDIT_RESCALE) c = tcoef[src];
            }
        }
        out_idx[o] = i;
        out_coef[o] = c;
    }
}

// Variance loss, without global atomics.
//  * Features below S (the index range of the low levels, S <= kVarSmallMax)
//    are hit by many slots of every token: each workgroup counts them in LDS
//    over a fixed range of tokens and writes one dense partial row; folds add
//    the rows in a fixed order.
//    Two passes (sums, then squared deviations about the mean) keep their
//    fp32 variance free of the cancellation of E[a^2] - E[a]^2.
//  * Features from S up are hit a few times per batch.  Their slots are
//    counting-sorted into buckets of 2^bsh consecutive features (bucket
//    histograms per workgroup, scans, a scatter of (feature, coefficient,
//    slot) records), then one workgroup per bucket accumulates counts and
//    fp64 sums of a and a^2 in LDS, one pass.
// Every slot gets a pre-gradient (a - mean) / count (0 outside F) in the
// workspace, so the gradient is one scaling pass; the sum over features is
// reduced in fp64 in a fixed order.
constexpr int kVarGroups = 256;        // workgroups of the passes over the code
constexpr int kVarThreads = 512;
constexpr int kVarSmallMax = 4096;     // LDS: up to 16 bytes per small feature
constexpr int kVarMinBucketShift = 10;
constexpr int kVarMaxBucketShift = 12;
constexpr int kVarBucket = 1 << kVarMaxBucketShift;   // LDS: 12 bytes per feature
constexpr int kVarMaxBuckets = 4096;   // LDS histogram of the scatter passes
constexpr int kVarBatch = 8;           // slots per lane loaded together

struct FeatStat {
    uint32_t cnt;
    float mean;
    float w;        // 1 / count for features in F, else 0
};

struct VarRed {
    double sum;
    unsigned long long cnt;
};

struct VarRec {
    int32_t feat;
    float a;
    int32_t slot;
};

struct VarWs {
    uint32_t* pcnt;     // [kVarGroups][S] partial counts of the small features
    float* pval;        // [kVarGroups][S] partial sums, then partial squared deviations
    FeatStat* small;    // [S]
    uint32_t* bcnt;     // [NB][kVarGroups] bucket counts, then offsets within the bucket
    uint32_t* btot;     // [NB]
    uint32_t* bstart;   // [NB]
    VarRed* red;        // [ceil(S / 16) + NB]
    VarRed* out;        // {sum of variances, |F|}
    VarRec* rec;        // [T k] slots of the features >= S, grouped by bucket
    float* pre;         // [T k] (a - mean) / count, 0 outside F
};

__host__ __device__ inline size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Buckets of 2^bsh features: the smallest shift >= kVarMinBucketShift that
// keeps the number of buckets within kVarMaxBuckets (none fits past
// kVarMaxBucketShift).
__host__ __device__ inline int var_bucket_shift(int64_t nfeat, int S)
{
    int sh = kVarMinBucketShift;
    while (sh < kVarMaxBucketShift && ((nfeat - S + (1 << sh) - 1) >> sh) > kVarMaxBuckets) ++sh;
    return sh;
}

__host__ __device__ inline int var_buckets(int64_t nfeat, int S)
{
    const int sh = var_bucket_shift(nfeat, S);
    return (int)((nfeat - S + (1 << sh) - 1) >> sh);
}

__host__ __device__ inline int var_small_blocks(int S) { return (S + 15) / 16; }

constexpr int kVarParts = 10;

// Byte offsets of the workspace parts; off[kVarParts] is the total size.
__host__ __device__ inline void var_offsets(int64_t nfeat, int S, int64_t nslots, size_t (&off)[kVarParts + 1])
{
    const int NB = var_buckets(nfeat, S);
    const size_t n4 = (size_t)nslots * 4;
    const size_t sz[kVarParts] = {(size_t)kVarGroups * S * 4, (size_t)kVarGroups * S * 4,
                                  (size_t)S * sizeof(FeatStat), (size_t)NB * kVarGroups * 4, (size_t)NB * 4,
                                  (size_t)NB * 4, (size_t)(var_small_blocks(S) + NB) * sizeof(VarRed), 256,
                                  (size_t)nslots * sizeof(VarRec), n4};
    off[0] = 0;
    for (int j = 0; j < kVarParts; ++j) off[j + 1] = off[j] + align256(sz[j]);
}

__host__ __device__ inline VarWs var_ws(void* ws, int64_t nfeat, int S, int64_t nslots)
{
    unsigned char* b = (unsigned char*)ws;
    size_t off[kVarParts + 1];
    var_offsets(nfeat, S, nslots, off);
    VarWs W;
    W.pcnt = (uint32_t*)(b + off[0]);
    W.pval = (float*)(b + off[1]);
    W.small = (FeatStat*)(b + off[2]);
    W.bcnt = (uint32_t*)(b + off[3]);
    W.btot = (uint32_t*)(b + off[4]);
    W.bstart = (uint32_t*)(b + off[5]);
    W.red = (VarRed*)(b + off[6]);
    W.out = (VarRed*)(b + off[7]);
    W.rec = (VarRec*)(b + off[8]);
    W.pre = (float*)(b + off[9]);
    return W;
}

// Tokens [t0, t1) of workgroup g of kVarGroups.
__device__ __forceinline__ void var_range(int64_t T, int64_t& t0, int64_t& t1)
{
    t0 = T * blockIdx.x / kVarGroups;
    t1 = T * (blockIdx.x + 1) / kVarGroups;
}

// Pass 1 over the code: small-feature counts and sums in LDS, and the bucket
// histogram of the other slots.
__global__ __launch_bounds__(kVarThreads) void var_count_kernel(const int32_t* idx, const float* coef, int64_t T, int k,
                                                                int64_t nfeat, int S, VarWs W)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int NB = var_buckets(nfeat, S), bsh = var_bucket_shift(nfeat, S);
    uint32_t* lcnt = (uint32_t*)smem;
    float* lsum = (float*)(smem + 4 * (size_t)S);
    uint32_t* hist = (uint32_t*)(smem + 8 * (size_t)S);
    for (int f = threadIdx.x; f < S; f += kVarThreads) {
        lcnt[f] = 0u;
        lsum[f] = 0.f;
    }
    for (int b = threadIdx.x; b < NB; b += kVarThreads) hist[b] = 0u;
    __syncthreads();
    int64_t t0, t1;
    var_range(T, t0, t1);
    const int64_t s1 = t1 * k;
    for (int64_t s0 = t0 * k + threadIdx.x; s0 < s1; s0 += kVarThreads * kVarBatch) {
        int32_t iv[kVarBatch];
#pragma unroll
        for (int b = 0; b < kVarBatch; ++b) {
            const int64_t s = s0 + (int64_t)b * kVarThreads;
            iv[b] = s < s1 ? idx[s] : -1;
        }
#pragma unroll
        for (int b = 0; b < kVarBatch; ++b) {
            const int32_t i = iv[b];
            if (i >= 0 && i < S) {
                atomicAdd(&lcnt[i], 1u);
                atomicAdd(&lsum[i], coef[s0 + (int64_t)b * kVarThreads]);
            } else if (i >= S && (int64_t)i < nfeat) {
                atomicAdd(&hist[(i - S) >> bsh], 1u);
            }
        }
    }
    __syncthreads();
    const int64_t row = (int64_t)blockIdx.x * S;
    for (int f = threadIdx.x; f < S; f += kVarThreads) {
        W.pcnt[row + f] = lcnt[f];
        W.pval[row + f] = lsum[f];
    }
    for (int b = threadIdx.x; b < NB; b += kVarThreads) W.bcnt[(int64_t)b * kVarGroups + blockIdx.x] = hist[b];
}

// Small features: counts and means from the partial rows (16 features x 16
// slices of the groups per block, fixed order); w = 1 / count for F.
__global__ __launch_bounds__(256) void var_small_stats_kernel(int S, int n_min, VarWs W)
{
    __shared__ uint32_t sc[16][17];
    __shared__ float sv[16][17];
    const int fl = threadIdx.x & 15, slice = threadIdx.x >> 4;
    const int f = blockIdx.x * 16 + fl;
    uint32_t c = 0;
    float v = 0.f;
    if (f < S)
        for (int g = slice; g < kVarGroups; g += 16) {
            c += W.pcnt[(int64_t)g * S + f];
            v += W.pval[(int64_t)g * S + f];
        }
    sc[slice][fl] = c;
    sv[slice][fl] = v;
    __syncthreads();
    if (slice == 0 && f < S) {
        for (int j = 1; j < 16; ++j) {
            c += sc[j][fl];
            v += sv[j][fl];
        }
        const bool inF = c > 0 && (int64_t)c >= (int64_t)n_min;
        W.small[f] = FeatStat{c, c ? v / (float)c : 0.f, inF ? 1.f / (float)c : 0.f};
    }
}

// Exclusive scan of each bucket's counts over the groups (one wave per bucket).
__global__ __launch_bounds__(256) void var_bucket_offsets_kernel(int NB, VarWs W)
{
    static_assert(kVarGroups == 256, "4 groups per lane");
    const int b = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
    if (b >= NB) return;
    uint32_t* c = W.bcnt + (int64_t)b * kVarGroups + lane * 4;
    const uint32_t c0 = c[0], c1 = c[1], c2 = c[2], c3 = c[3];
    const uint32_t own = c0 + c1 + c2 + c3;
    uint32_t incl = own;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const uint32_t v = __shfl_up(incl, off, 64);
        if (lane >= off) incl += v;
    }
    const uint32_t ex = incl - own;
    c[0] = ex;
    c[1] = ex + c0;
    c[2] = ex + c0 + c1;
    c[3] = ex + c0 + c1 + c2;
    if (lane == 63) W.btot[b] = incl;
}

// Exclusive scan of the bucket totals (one block, any NB).
__global__ __launch_bounds__(1024) void var_bucket_starts_kernel(int NB, VarWs W)
{
    __shared__ uint32_t wsum[16];
    __shared__ uint32_t carry;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (threadIdx.x == 0) carry = 0;
    __syncthreads();
    for (int base = 0; base < NB; base += 1024) {
        const int b = base + threadIdx.x;
        const uint32_t v = b < NB ? W.btot[b] : 0u;
        uint32_t incl = v;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const uint32_t u = __shfl_up(incl, off, 64);
            if (lane >= off) incl += u;
        }
        if (lane == 63) wsum[wave] = incl;
        __syncthreads();
        uint32_t before = carry;
        for (int j = 0; j < wave; ++j) before += wsum[j];
        if (b < NB) W.bstart[b] = before + incl - v;
        __syncthreads();
        if (threadIdx.x == 1023) carry = before + incl;
        __syncthreads();
    }
}

// Pass 2 over the code: squared deviations of the small features in LDS and
// their pre-gradients; the other slots are scattered into their buckets.
__global__ __launch_bounds__(kVarThreads) void var_scatter_kernel(const int32_t* idx, const float* coef, int64_t T,
                                                                  int k, int64_t nfeat, int S, VarWs W)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int NB = var_buckets(nfeat, S), bsh = var_bucket_shift(nfeat, S);
    float* lmean = (float*)smem;
    float* lw = (float*)(smem + 4 * (size_t)S);
    float* lsq = (float*)(smem + 8 * (size_t)S);
    uint32_t* cursor = (uint32_t*)(smem + 12 * (size_t)S);
    for (int f = threadIdx.x; f < S; f += kVarThreads) {
        const FeatStat st = W.small[f];
        lmean[f] = st.mean;
        lw[f] = st.w;
        lsq[f] = 0.f;
    }
    for (int b = threadIdx.x; b < NB; b += kVarThreads)
        cursor[b] = W.bstart[b] + W.bcnt[(int64_t)b * kVarGroups + blockIdx.x];
    __syncthreads();
    int64_t t0, t1;
    var_range(T, t0, t1);
    const int64_t s1 = t1 * k;
    for (int64_t s0 = t0 * k + threadIdx.x; s0 < s1; s0 += kVarThreads * kVarBatch) {
        int32_t iv[kVarBatch];
        float av[kVarBatch];
#pragma unroll
        for (int b = 0; b < kVarBatch; ++b) {
            const int64_t s = s0 + (int64_t)b * kVarThreads;
            iv[b] = s < s1 ? idx[s] : INT32_MIN;
        }
#pragma unroll
        for (int b = 0; b < kVarBatch; ++b) {
            const int32_t i = iv[b];
            av[b] = (i >= 0 && (int64_t)i < nfeat) ? coef[s0 + (int64_t)b * kVarThreads] : 0.f;
        }
#pragma unroll
        for (int b = 0; b < kVarBatch; ++b) {
            const int32_t i = iv[b];
            if (i == INT32_MIN) continue;
            const int64_t s = s0 + (int64_t)b * kVarThreads;
            if (i >= 0 && i < S) {
                const float dv = av[b] - lmean[i];
                atomicAdd(&lsq[i], dv * dv);
                W.pre[s] = lw[i] * dv;
            } else if (i >= S && (int64_t)i < nfeat) {
                const uint32_t p = atomicAdd(&cursor[(i - S) >> bsh], 1u);
                W.rec[p] = VarRec{i, av[b], (int32_t)s};
            } else {
                W.pre[s] = 0.f;
            }
        }
    }
    __syncthreads();
    const int64_t row = (int64_t)blockIdx.x * S;
    for (int f = threadIdx.x; f < S; f += kVarThreads) W.pval[row + f] = lsq[f];
}

// Small features: squared deviations from the partial rows; each block's
// variance sum and |F| count go to its reduction entry.
__global__ __launch_bounds__(256) void var_small_var_kernel(int S, VarWs W)
{
    __shared__ float sv[16][17];
    const int fl = threadIdx.x & 15, slice = threadIdx.x >> 4;
    const int f = blockIdx.x * 16 + fl;
    float v = 0.f;
    if (f < S)
        for (int g = slice; g < kVarGroups; g += 16) v += W.pval[(int64_t)g * S + f];
    sv[slice][fl] = v;
    __syncthreads();
    if (threadIdx.x == 0) {
        double sum = 0.0;
        unsigned long long cnt = 0;
        for (int j = 0; j < 16; ++j) {
            const int ff = blockIdx.x * 16 + j;
            if (ff >= S) break;
            float q = 0.f;
            for (int sl = 0; sl < 16; ++sl) q += sv[sl][j];
            const FeatStat st = W.small[ff];
            if (st.w > 0.f) {
                sum += (double)q / (double)st.cnt;
                ++cnt;
            }
        }
        W.red[blockIdx.x] = VarRed{sum, cnt};
    }
}

// One workgroup per bucket of 2^bsh features: count, sum and sum of squares
// per feature in LDS (the sums in fp64, so that E[a^2] - E[a]^2 keeps its
// precision for fp32 data); the bucket's variance sum and |F| count; and the
// pre-gradient of each of its slots.  Each lane keeps kVarBatch records in
// flight per round.
constexpr int kVarBucketThreads = 1024;

template <typename F>
__device__ __forceinline__ void var_bucket_loop(const VarRec* rec, int64_t p0, int64_t p1, int32_t f0, F f)
{
    for (int64_t q0 = p0 + threadIdx.x; q0 < p1; q0 += (int64_t)kVarBucketThreads * kVarBatch) {
        VarRec r[kVarBatch];
#pragma unroll
        for (int j = 0; j < kVarBatch; ++j) {
            const int64_t q = q0 + (int64_t)j * kVarBucketThreads;
            r[j] = q < p1 ? rec[q] : VarRec{f0 - 1, 0.f, 0};
        }
#pragma unroll
        for (int j = 0; j < kVarBatch; ++j)
            if (r[j].feat >= f0) f(r[j].feat - f0, r[j].a, r[j].slot);
    }
}

__global__ __launch_bounds__(kVarBucketThreads) void var_bucket_kernel(int64_t nfeat, int S, int bsh, int n_min,
                                                                       VarWs W)
{
    (void)nfeat;   // buckets cover [S, nfeat) by construction of the grid
    extern __shared__ __align__(16) unsigned char smem[];
    __shared__ double rs[kVarBucketThreads / 64];
    __shared__ unsigned long long rc[kVarBucketThreads / 64];
    const int b = blockIdx.x, nf = 1 << bsh;
    double* s1 = (double*)smem;                       // sums, then means
    double* s2 = s1 + nf;                             // sums of squares
    uint32_t* lcnt = (uint32_t*)(s2 + nf);
    float* lmean = (float*)s2;                        // after the reduction: mean,
    float* lw = lmean + nf;                           // and weight w
    const int32_t f0 = (int32_t)(S + ((int64_t)b << bsh));
    for (int f = threadIdx.x; f < nf; f += kVarBucketThreads) {
        s1[f] = 0.0;
        s2[f] = 0.0;
        lcnt[f] = 0u;
    }
    __syncthreads();
    const int64_t p0 = W.bstart[b], p1 = p0 + W.btot[b];
    var_bucket_loop(W.rec, p0, p1, f0, [&](int f, float a, int) {
        atomicAdd(&lcnt[f], 1u);
        atomicAdd(&s1[f], (double)a);
        atomicAdd(&s2[f], (double)a * (double)a);
    });
    __syncthreads();
    double v = 0.0;
    unsigned long long c = 0;
    float mv[kVarBucket / kVarBucketThreads], wv[kVarBucket / kVarBucketThreads];
#pragma unroll
    for (int j = 0; j < kVarBucket / kVarBucketThreads; ++j) {
        const int f = threadIdx.x + j * kVarBucketThreads;
        mv[j] = 0.f;
        wv[j] = 0.f;
        if (f >= nf) continue;
        const uint32_t n = lcnt[f];
        if (n == 0) continue;
        const double mean = s1[f] / (double)n;
        const bool inF = (int64_t)n >= (int64_t)n_min;
        if (inF) {
            v += fmax(s2[f] / (double)n - mean * mean, 0.0);
            ++c;
        }
        mv[j] = (float)mean;
        wv[j] = inF ? 1.f / (float)n : 0.f;
    }
    __syncthreads();      // s2 is overwritten by the float mean / weight tables
#pragma unroll
    for (int j = 0; j < kVarBucket / kVarBucketThreads; ++j) {
        const int f = threadIdx.x + j * kVarBucketThreads;
        if (f < nf) {
            lmean[f] = mv[j];
            lw[f] = wv[j];
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        v += __shfl_xor(v, off, 64);
        c += __shfl_xor(c, off, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        rs[threadIdx.x >> 6] = v;
        rc[threadIdx.x >> 6] = c;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double sv = 0.0;
        unsigned long long sc = 0;
        for (int j = 0; j < kVarBucketThreads / 64; ++j) {
            sv += rs[j];
            sc += rc[j];
        }
        W.red[var_small_blocks(S) + b] = VarRed{sv, sc};
    }
    var_bucket_loop(W.rec, p0, p1, f0, [&](int f, float a, int slot) { W.pre[slot] = lw[f] * (a - lmean[f]); });
}

// The loss from the nred reduction entries, summed in a fixed order.
__global__ __launch_bounds__(256) void var_final_kernel(int nred, VarWs W, float* loss)
{
    __shared__ double ps[4];
    __shared__ unsigned long long pc[4];
    double v = 0.0;
    unsigned long long c = 0;
    for (int j = threadIdx.x; j < nred; j += 256) {
        v += W.red[j].sum;
        c += W.red[j].cnt;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        v += __shfl_xor(v, off, 64);
        c += __shfl_xor(c, off, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        ps[threadIdx.x >> 6] = v;
        pc[threadIdx.x >> 6] = c;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        const double sv = ps[0] + ps[1] + ps[2] + ps[3];
        const unsigned long long sc = pc[0] + pc[1] + pc[2] + pc[3];
        W.out->sum = sv;
        W.out->cnt = sc;
        *loss = sc ? (float)(-sv / (double)sc) : 0.f;
    }
}

// grad = scale * -(2/|F|) * pre-gradient.
__global__ void var_grad_kernel(int64_t n, VarWs W, float* grad, const float* grad_scale)
{
    const unsigned long long F = W.out->cnt;
    const float w = F ? (grad_scale ? *grad_scale : 1.f) * (-2.f / (float)F) : 0.f;
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < n; s += (int64_t)gridDim.x * blockDim.x)
        grad[s] = w * W.pre[s];
}

int device_cus_x()
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

dim3 row_grid(int64_t T)
{
    const int64_t need = (T + kRowWaves - 1) / kRowWaves;
    return dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, (int64_t)device_cus_x() * 8)));
}

// Register chunks of 512 elements per row: 1, 2 or 4 (d <= 2048), else 0.
int row_chunks(int d)
{
    const int c = (d + 511) / 512;
    return c <= 1 ? 1 : c == 2 ? 2 : c <= 4 ? 4 : 0;
}

dim3 flat_grid(int64_t n, int threads)
{
    const int64_t need = (n + threads - 1) / threads;
    return dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, (int64_t)device_cus_x() * 16)));
}

}  // namespace

hipError_t launch_normalize(int d, int64_t T, const void* u, bool u16, const void* ref, bool r16,
                            const int32_t* ref_rows, int64_t T_ref, void* y, bool y16, float* norms,
                            hipStream_t stream)
{
    RowIO io{u, u16, ref, r16, nullptr, false, y, y16, nullptr, false};
    const dim3 grid = row_grid(T), block(kRowThreads);
    switch (row_chunks(d)) {
    case 1: hipLaunchKernelGGL(normalize_kernel<1>, grid, block, 0, stream, io, d, T, ref_rows, T_ref, norms); break;
    case 2: hipLaunchKernelGGL(normalize_kernel<2>, grid, block, 0, stream, io, d, T, ref_rows, T_ref, norms); break;
    case 4: hipLaunchKernelGGL(normalize_kernel<4>, grid, block, 0, stream, io, d, T, ref_rows, T_ref, norms); break;
    default: hipLaunchKernelGGL(normalize_kernel<0>, grid, block, 0, stream, io, d, T, ref_rows, T_ref, norms); break;
    }
    return hipGetLastError();
}

hipError_t launch_normalize_bwd(int d, int64_t T, const void* g, bool g16, const void* u, bool u16, const void* ref,
                                bool r16, void* gu, bool gu16, void* gr, bool gr16, int accumulate, hipStream_t stream)
{
    RowIO io{g, g16, u, u16, ref, r16, gu, gu16, gr, gr16};
    const dim3 grid = row_grid(T), block(kRowThreads);
    switch (row_chunks(d)) {
    case 1: hipLaunchKernelGGL(normalize_bwd_kernel<1>, grid, block, 0, stream, io, d, T, accumulate); break;
    case 2: hipLaunchKernelGGL(normalize_bwd_kernel<2>, grid, block, 0, stream, io, d, T, accumulate); break;
    case 4: hipLaunchKernelGGL(normalize_bwd_kernel<4>, grid, block, 0, stream, io, d, T, accumulate); break;
    default: hipLaunchKernelGGL(normalize_bwd_kernel<0>, grid, block, 0, stream, io, d, T, accumulate); break;
    }
    return hipGetLastError();
}

hipError_t launch_edit_codes(const int32_t* idx, const float* coef, const int32_t* tidx, const float* tcoef,
                             int64_t T, int k, const int32_t* rows, const int32_t* slots, const int32_t* ops,
                             int64_t E, int32_t* out_idx, float* out_coef, hipStream_t stream)
{
    hipLaunchKernelGGL(edit_kernel, flat_grid(E * k, 256), dim3(256), 0, stream, idx, coef, tidx, tcoef, T, k, rows,
                       slots, ops, E, out_idx, out_coef);
    return hipGetLastError();
}

// Index range of the levels counted in LDS: 2^{n_l} of the highest level l
// with 2^{n_l} <= kVarSmallMax (0 when even level 0 is larger).
int variance_small_range(const int* level_bits, int levels)
{
    int S = 0;
    for (int l = 0; l < levels; ++l)
        if ((1 << level_bits[l]) <= kVarSmallMax) S = 1 << level_bits[l];
    return S;
}

bool variance_supported(int64_t nfeat, int S, int64_t nslots)
{
    return var_buckets(nfeat, S) <= kVarMaxBuckets && nslots < ((int64_t)1 << 31);
}

size_t variance_workspace_bytes(int64_t nfeat, int S, int64_t nslots)
{
    size_t off[kVarParts + 1];
    var_offsets(nfeat, S, nslots, off);
    return off[kVarParts];
}

hipError_t launch_variance_loss(const int32_t* idx, const float* coef, int64_t T, int k, int64_t nfeat, int S,
                                int n_min, void* ws, float* loss, float* grad, const float* grad_scale,
                                hipStream_t stream)
{
    const int64_t n = T * k;
    const VarWs W = var_ws(ws, nfeat, S, n);
    const int NB = var_buckets(nfeat, S);
    const dim3 groups(kVarGroups), threads(kVarThreads);
    const int SB = var_small_blocks(S);
    const size_t lds_count = 8 * (size_t)S + 4 * (size_t)NB, lds_scatter = 12 * (size_t)S + 4 * (size_t)NB;
    allow_lds(var_count_kernel, lds_count);
    allow_lds(var_scatter_kernel, lds_scatter);
    hipLaunchKernelGGL(var_count_kernel, groups, threads, lds_count, stream, idx, coef, T, k, nfeat, S, W);
    if (S > 0) hipLaunchKernelGGL(var_small_stats_kernel, dim3(SB), dim3(256), 0, stream, S, n_min, W);
    if (NB > 0) {
        hipLaunchKernelGGL(var_bucket_offsets_kernel, dim3((NB + 3) / 4), dim3(256), 0, stream, NB, W);
        hipLaunchKernelGGL(var_bucket_starts_kernel, dim3(1), dim3(1024), 0, stream, NB, W);
    }
    hipLaunchKernelGGL(var_scatter_kernel, groups, threads, lds_scatter, stream, idx, coef, T, k, nfeat, S, W);
    if (S > 0) hipLaunchKernelGGL(var_small_var_kernel, dim3(SB), dim3(256), 0, stream, S, W);
    if (NB > 0) {
        const int bsh = var_bucket_shift(nfeat, S);
        const size_t lds_bucket = (size_t)20 << bsh;
        allow_lds(var_bucket_kernel, lds_bucket);
        hipLaunchKernelGGL(var_bucket_kernel, dim3(NB), dim3(kVarBucketThreads), lds_bucket, stream, nfeat, S, bsh,
                           n_min, W);
    }
    hipLaunchKernelGGL(var_final_kernel, dim3(1), dim3(256), 0, stream, SB + NB, W, loss);
    if (grad && n > 0)
        hipLaunchKernelGGL(var_grad_kernel, flat_grid(n, 256), dim3(256), 0, stream, n, W, grad, grad_scale);
    return hipGetLastError();
}

hipError_t launch_variance_grad(int64_t T, int k, int64_t nfeat, int S, void* ws, float* grad,
                                const float* grad_scale, hipStream_t stream)
{
    const int64_t n = T * k;
    const VarWs W = var_ws(ws, nfeat, S, n);
    if (n > 0) hipLaunchKernelGGL(var_grad_kernel, flat_grid(n, 256), dim3(256), 0, stream, n, W, grad, grad_scale);
    return hipGetLastError();
}

}  // namespace dpb
