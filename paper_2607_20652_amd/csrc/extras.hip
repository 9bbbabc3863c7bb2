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
            q.x = f32_to_bf16_rne(v[0]) | (f32_to_bf16_rne(v[1]) << 16);
            q.y = f32_to_bf16_rne(v[2]) | (f32_to_bf16_rne(v[3]) << 16);
            q.z = f32_to_bf16_rne(v[4]) | (f32_to_bf16_rne(v[5]) << 16);
            q.w = f32_to_bf16_rne(v[6]) | (f32_to_bf16_rne(v[7]) << 16);
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

// y = u * ||ref|| / ||u|| per row (0 when ||u|| = 0); norms[t] = (||ref||, ||u||).
// Row t's reference is row ref_rows[t] of ref when ref_rows is given (norm 0
// when that index is outside [0, T_ref)).
__global__ __launch_bounds__(kRowThreads) void normalize_kernel(RowIO io, int d, int64_t T, const int32_t* ref_rows,
                                                                int64_t T_ref, float* norms)
{
    const int lane = threadIdx.x & 63;
    const bool vec = (d & 7) == 0;
    for (int64_t t = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6); t < T; t += (int64_t)gridDim.x * kRowWaves) {
        const int64_t r0 = t * d;
        const int64_t rr = ref_rows ? (int64_t)ref_rows[t] : t;
        const bool has_ref = rr >= 0 && rr < T_ref;
        const int64_t q0 = has_ref ? rr * d : 0;
        float su = 0.f, sr = 0.f;
        for (int o = lane * 8; o < d; o += 512) {
            float u[8], r[8];
            load8(io.a, io.a16, r0 + o, r0 + d, vec, u);
#pragma unroll
            for (int e = 0; e < 8; ++e) su += u[e] * u[e];
            if (has_ref) {
                load8(io.b, io.b16, q0 + o, q0 + d, vec, r);
#pragma unroll
                for (int e = 0; e < 8; ++e) sr += r[e] * r[e];
            }
        }
        su = wave_sum(su);
        sr = wave_sum(sr);
        const float nu = sqrtf(su), nr = sqrtf(sr);
        const float scale = nu > 0.f ? nr / nu : 0.f;
        for (int o = lane * 8; o < d; o += 512) {
            float u[8];
            load8(io.a, io.a16, r0 + o, r0 + d, vec, u);
#pragma unroll
            for (int e = 0; e < 8; ++e) u[e] *= scale;
            store8(io.o1, io.o116, r0 + o, r0 + d, vec, u);
        }
        if (lane == 0 && norms) {
            norms[2 * t] = nr;
            norms[2 * t + 1] = nu;
        }
    }
}

// grad_u = s (g - (<g,u>/||u||^2) u), grad_ref (+)= (<g,u> / (||u|| ||ref||)) ref.
__global__ __launch_bounds__(kRowThreads) void normalize_bwd_kernel(RowIO io, int d, int64_t T, int accumulate)
{
    const int lane = threadIdx.x & 63;
    const bool vec = (d & 7) == 0;
    for (int64_t t = (int64_t)blockIdx.x * kRowWaves + (threadIdx.x >> 6); t < T; t += (int64_t)gridDim.x * kRowWaves) {
        const int64_t r0 = t * d;
        float su = 0.f, sr = 0.f, gu = 0.f;
        for (int o = lane * 8; o < d; o += 512) {
            float g[8], u[8], r[8];
            load8(io.a, io.a16, r0 + o, r0 + d, vec, g);
            load8(io.b, io.b16, r0 + o, r0 + d, vec, u);
            load8(io.c, io.c16, r0 + o, r0 + d, vec, r);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                su += u[e] * u[e];
                sr += r[e] * r[e];
                gu += g[e] * u[e];
            }
        }
        su = wave_sum(su);
        sr = wave_sum(sr);
        gu = wave_sum(gu);
        const float nu = sqrtf(su), nr = sqrtf(sr);
        const float s = nu > 0.f ? nr / nu : 0.f;
        const float cu = nu > 0.f ? s * gu / su : 0.f;
        const float cr = (nu > 0.f && nr > 0.f) ? gu / (nu * nr) : 0.f;
        for (int o = lane * 8; o < d; o += 512) {
            float g[8], u[8], r[8], a[8];
            load8(io.a, io.a16, r0 + o, r0 + d, vec, g);
            load8(io.b, io.b16, r0 + o, r0 + d, vec, u);
            load8(io.c, io.c16, r0 + o, r0 + d, vec, r);
#pragma unroll
            for (int e = 0; e < 8; ++e) u[e] = s * g[e] - cu * u[e];
            store8(io.o1, io.o116, r0 + o, r0 + d, vec, u);
            if (accumulate) load8(io.o2, io.o216, r0 + o, r0 + d, vec, a);
#pragma unroll
            for (int e = 0; e < 8; ++e) a[e] = (accumulate ? a[e] : 0.f) + cr * r[e];
            store8(io.o2, io.o216, r0 + o, r0 + d, vec, a);
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

// Variance loss workspace: per feature {count: u32, sum: f32, squared
// deviations: f32}, then {sum of variances: f64, |F|: u64}.  Two passes over
// the code (sums, then squared deviations about the mean) keep the variance
// free of the cancellation of E[a^2] - E[a]^2.
struct FeatStat {
    uint32_t cnt;
    float sum;
    float sq;
};

__global__ void fill_zero_kernel(uint32_t* p, int64_t n)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) p[i] = 0u;
}

__global__ void feature_sums_kernel(const int32_t* idx, const float* coef, int64_t n, int64_t nfeat, FeatStat* tab)
{
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < n; s += (int64_t)gridDim.x * blockDim.x) {
        const int32_t i = idx[s];
        if (i < 0 || (int64_t)i >= nfeat) continue;
        atomicAdd(&tab[i].cnt, 1u);
        atomicAdd(&tab[i].sum, coef[s]);
    }
}

__global__ void feature_sqdev_kernel(const int32_t* idx, const float* coef, int64_t n, int64_t nfeat, FeatStat* tab)
{
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < n; s += (int64_t)gridDim.x * blockDim.x) {
        const int32_t i = idx[s];
        if (i < 0 || (int64_t)i >= nfeat) continue;
        const float dv = coef[s] - tab[i].sum / (float)tab[i].cnt;
        atomicAdd(&tab[i].sq, dv * dv);
    }
}

// Features with count >= n_min: their variance into the fp64 sum and +1 to
// |F|; (mean, 1/count) are left in the table for the gradient, and the count
// of a feature outside F is cleared.
__global__ __launch_bounds__(256) void variance_reduce_kernel(FeatStat* tab, int64_t nfeat, int n_min, double* acc,
                                                              unsigned long long* nF)
{
    double v = 0.0;
    unsigned long long c = 0;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nfeat; i += (int64_t)gridDim.x * blockDim.x) {
        const uint32_t cnt = tab[i].cnt;
        if (cnt == 0) continue;
        if ((int64_t)cnt >= (int64_t)n_min) {
            v += (double)tab[i].sq / (double)cnt;
            ++c;
            tab[i].sum = tab[i].sum / (float)cnt;
            tab[i].sq = 1.f / (float)cnt;
        } else {
            tab[i].cnt = 0;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
        v += __shfl_xor(v, off, 64);
        c += __shfl_xor(c, off, 64);
    }
    if ((threadIdx.x & 63) == 0) {
        atomicAdd(acc, v);
        atomicAdd(nF, c);
    }
}

// loss = -(1/|F|) sum of variances; grad = scale * -(2/|F|) (a - mean) / count.
__global__ void variance_grad_kernel(const int32_t* idx, const float* coef, int64_t n, int64_t nfeat,
                                     const FeatStat* tab, const double* acc, const unsigned long long* nF,
                                     float* loss, float* grad, const float* grad_scale)
{
    const unsigned long long F = *nF;
    if (blockIdx.x == 0 && threadIdx.x == 0) *loss = F ? (float)(-*acc / (double)F) : 0.f;
    if (!grad) return;
    const float w = F ? (grad_scale ? *grad_scale : 1.f) * (-2.f / (float)F) : 0.f;
    for (int64_t s = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; s < n; s += (int64_t)gridDim.x * blockDim.x) {
        const int32_t i = idx[s];
        float gr = 0.f;
        if (i >= 0 && (int64_t)i < nfeat && tab[i].cnt) gr = w * (coef[s] - tab[i].sum) * tab[i].sq;
        grad[s] = gr;
    }
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
    hipLaunchKernelGGL(normalize_kernel, row_grid(T), dim3(kRowThreads), 0, stream, io, d, T, ref_rows, T_ref, norms);
    return hipGetLastError();
}

hipError_t launch_normalize_bwd(int d, int64_t T, const void* g, bool g16, const void* u, bool u16, const void* ref,
                                bool r16, void* gu, bool gu16, void* gr, bool gr16, int accumulate, hipStream_t stream)
{
    RowIO io{g, g16, u, u16, ref, r16, gu, gu16, gr, gr16};
    hipLaunchKernelGGL(normalize_bwd_kernel, row_grid(T), dim3(kRowThreads), 0, stream, io, d, T, accumulate);
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

size_t variance_workspace_bytes(int64_t nfeat)
{
    return (((size_t)nfeat * sizeof(FeatStat) + 15) & ~(size_t)15) + 32;
}

hipError_t launch_variance_loss(const int32_t* idx, const float* coef, int64_t n, int64_t nfeat, int n_min,
                                void* ws, float* loss, float* grad, const float* grad_scale, hipStream_t stream)
{
    FeatStat* tab = (FeatStat*)ws;
    const size_t tab_bytes = ((size_t)nfeat * sizeof(FeatStat) + 15) & ~(size_t)15;
    double* acc = (double*)((unsigned char*)ws + tab_bytes);
    unsigned long long* nF = (unsigned long long*)((unsigned char*)ws + tab_bytes + 8);
    const int64_t words = (int64_t)(tab_bytes + 16) / 4;
    const dim3 b(256);
    hipLaunchKernelGGL(fill_zero_kernel, flat_grid(words, 256), b, 0, stream, (uint32_t*)ws, words);
    if (n > 0) {
        hipLaunchKernelGGL(feature_sums_kernel, flat_grid(n, 256), b, 0, stream, idx, coef, n, nfeat, tab);
        hipLaunchKernelGGL(feature_sqdev_kernel, flat_grid(n, 256), b, 0, stream, idx, coef, n, nfeat, tab);
    }
    hipLaunchKernelGGL(variance_reduce_kernel, flat_grid(nfeat, 256), b, 0, stream, tab, nfeat, n_min, acc, nF);
    hipLaunchKernelGGL(variance_grad_kernel, flat_grid(n, 256), b, 0, stream, idx, coef, n, nfeat, tab, acc, nF, loss,
                       grad, grad_scale);
    return hipGetLastError();
}

}  // namespace dpb
