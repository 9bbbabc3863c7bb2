// EMA statistics of the score standardization (§2.2 "Score
// Standardization") for gfx950.
//
// State, owned by the caller: stats[N] = (mu, r = 1/sigma) as float2, read by
// the encoder, and m2[N] (the EMA of the second raw moment).  After a batch encoded
// with the state, the moments of each feature over the tokens where it was a
// candidate update it:
//  * level 0: a basis feature is a candidate at every token, so its sample is
//    a column of x over the whole batch -- per-workgroup fp64 column sums over
//    a fixed token range, folded in a fixed order;
//  * levels l >= 1: on kStdSample evenly spaced tokens, the children
//    p XOR g_j of the active parents (the level l-1 entries of the token's
//    code), each child once per token, scored on the matrix cores
//    (<phi_c, x> by the child-scoring contraction); one record per
//    (token, child).  Records of one feature are
//    combined with fp64 atomics in a per-feature accumulator that only the
//    records themselves clear, and the record with the lowest position
//    applies the update.
// Update of a feature with n samples s_1..s_n (moving averages of the first
// two raw moments, so that a feature sampled once per batch still measures
// its spread across batches):
//    mu <- (1 - beta) mu + beta mean(s),  m2 <- (1 - beta) m2 + beta mean(s^2),
//    r = 1 / sqrt(max(m2 - mu^2, 0) + eps).
#include <algorithm>

#include "scoring.hpp"

namespace dpb {
namespace {

constexpr int kStdGroups = 256;     // workgroups of the level-0 column pass
constexpr int kStdThreads = 256;

struct StdAcc {
    uint32_t n;
    uint32_t owner;
    double s1;
    double s2;
};

struct StdRec {
    int32_t feat;      // -1: none (duplicate child or missing parent)
    float s;
};

struct StdWs {
    double* col;       // [kStdGroups][d][2] fp64 column sums of x and x^2
    StdRec* rec;       // [kStdSample][cands]
    StdAcc* acc;       // [N]
};

__host__ __device__ inline size_t std_align(size_t v) { return (v + 255) & ~(size_t)255; }

__host__ __device__ inline int std_cands(const DevPlan& P)
{
    int c = 0;
    for (int l = 1; l < P.levels; ++l) c += P.active[l - 1] * P.delta[l];
    return c;
}

__host__ __device__ inline StdWs std_ws(void* ws, const DevPlan& P, size_t* total)
{
    unsigned char* b = (unsigned char*)ws;
    const int64_t N = (int64_t)1 << P.level_bits[P.levels - 1];
    const size_t o1 = std_align((size_t)kStdGroups * P.d * 16);
    const size_t o2 = o1 + std_align((size_t)kStdSample * std_cands(P) * sizeof(StdRec));
    const size_t o3 = o2 + std_align((size_t)N * sizeof(StdAcc));
    if (total) *total = o3;
    StdWs W{};
    if (!ws) return W;
    W.col = (double*)b;
    W.rec = (StdRec*)(b + o1);
    W.acc = (StdAcc*)(b + o2);
    return W;
}

__device__ __forceinline__ void ema(float2* stats, float* m2, int64_t c, double n, double s1, double s2, float beta,
                                    float eps)
{
    const float mu = (1.f - beta) * stats[c].x + beta * (float)(s1 / n);
    const float q = (1.f - beta) * m2[c] + beta * (float)(s2 / n);
    m2[c] = q;
    stats[c] = make_float2(mu, 1.f / sqrtf(fmaxf(q - mu * mu, 0.f) + eps));
}

__global__ void std_init_kernel(float2* stats, float* m2, int64_t N)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < N; i += (int64_t)gridDim.x * blockDim.x) {
        stats[i] = make_float2(0.f, 1.f);
        m2[i] = 1.f;
    }
}

// Column sums of x and x^2 over the tokens [T g / G, T (g + 1) / G) of
// workgroup g = blockIdx.x.  Each of its kStdColSlices slices sums a
// contiguous part of those rows, a thread four consecutive columns of a
// 1024-column strip (blockIdx.y), eight rows per round; the slices' sums are
// then added in slice order (a fixed order: the statistics do not depend on
// scheduling).
constexpr int kStdColSlices = 4;

template <bool BF16>
__global__ __launch_bounds__(kStdThreads * kStdColSlices) void std_col_kernel(const void* x, int d, int64_t T,
                                                                             StdWs W)
{
    __shared__ double part[kStdColSlices - 1][kStdThreads][8];
    const int slice = threadIdx.x / kStdThreads, tid = threadIdx.x % kStdThreads;
    const int c0 = blockIdx.y * 4 * kStdThreads + 4 * tid;
    const int64_t g0 = T * blockIdx.x / kStdGroups, g1 = T * (blockIdx.x + 1) / kStdGroups;
    const int64_t t0 = g0 + (g1 - g0) * slice / kStdColSlices, t1 = g0 + (g1 - g0) * (slice + 1) / kStdColSlices;
    const bool vec = (d & 3) == 0;
    double s1[4] = {0.0, 0.0, 0.0, 0.0}, s2[4] = {0.0, 0.0, 0.0, 0.0};
    if (c0 < d) {
        for (int64_t t = t0; t < t1; t += 8) {
            float v[8][4];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int64_t i = (t + e) * d + c0;
                if (t + e >= t1) {
#pragma unroll
                    for (int q = 0; q < 4; ++q) v[e][q] = 0.f;
                } else if (vec && BF16) {
                    const uint2 u = *(const uint2*)((const uint16_t*)x + i);
                    v[e][0] = bf16_bits_to_f32(u.x & 0xFFFFu);
                    v[e][1] = bf16_bits_to_f32(u.x >> 16);
                    v[e][2] = bf16_bits_to_f32(u.y & 0xFFFFu);
                    v[e][3] = bf16_bits_to_f32(u.y >> 16);
                } else if (vec) {
                    const float4 f = *(const float4*)((const float*)x + i);
                    v[e][0] = f.x; v[e][1] = f.y; v[e][2] = f.z; v[e][3] = f.w;
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q) v[e][q] = c0 + q < d ? load_act<BF16>(x, i + q) : 0.f;
                }
            }
#pragma unroll
            for (int e = 0; e < 8; ++e)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    s1[q] += (double)v[e][q];
                    s2[q] += (double)v[e][q] * (double)v[e][q];
                }
        }
    }
    if (slice > 0)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            part[slice - 1][tid][q] = s1[q];
            part[slice - 1][tid][4 + q] = s2[q];
        }
    __syncthreads();
    if (slice == 0 && c0 < d) {
#pragma unroll
        for (int sl = 0; sl < kStdColSlices - 1; ++sl)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                s1[q] += part[sl][tid][q];
                s2[q] += part[sl][tid][4 + q];
            }
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (c0 + q < d) {
                double* o = W.col + ((int64_t)blockIdx.x * d + c0 + q) * 2;
                o[0] = s1[q];
                o[1] = s2[q];
            }
    }
}

__global__ void std_col_update_kernel(int d, int64_t T, StdWs W, float2* stats, float* m2, float beta, float eps)
{
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    if (c >= d || T <= 0) return;
    double s1 = 0.0, s2 = 0.0;
    for (int g = 0; g < kStdGroups; ++g) {
        s1 += W.col[((int64_t)g * d + c) * 2];
        s2 += W.col[((int64_t)g * d + c) * 2 + 1];
    }
    ema(stats, m2, c, (double)T, s1, s2, beta, eps);
}

// One workgroup per (sampled token, level l >= 1, block of 16 parent slots
// of level l - 1): the scores <phi_c, x_t> of the children c = p XOR g_j of
// its parents, on the matrix cores (the encoder's child-scoring contraction
// of §2.2: generator tiles of Gamma_l against the sign-flipped row of x), one
// record per candidate.  A child reached from several parents is sampled once
// per token: every workgroup of the (token, level) inserts all of the level's
// candidates into an LDS hash set (linear probing, compare-and-swap; a
// child's slot ends up holding its lowest candidate position, so every
// workgroup of the token and level agrees on it), and a candidate is recorded
// only when it is that copy.
constexpr int kStdMaxCand = 8192;   // K_{l-1} Delta_l of the paper's 3-level hierarchy (32 x 256)

__host__ __device__ inline int std_hash_bits(const DevPlan& P)
{
    int n = 1;
    for (int l = 1; l < P.levels; ++l) n = std::max(n, P.active[l - 1] * P.delta[l]);
    int b = 8;
    while ((1 << b) < 2 * n) ++b;
    return b;
}

__host__ __device__ inline unsigned std_sample_lds(const DevPlan& P, bool x_bf16)
{
    return align16u(4u << std_hash_bits(P)) + align16u(x_bf16 ? P.prow * 4 : P.dp * 4) + align16u(16 * P.cws * 4);
}

__host__ __device__ inline int std_parent_blocks(const DevPlan& P)
{
    int nb = 1;
    for (int l = 1; l < P.levels; ++l) nb = std::max(nb, (P.active[l - 1] + 15) / 16);
    return nb;
}

__device__ __forceinline__ uint32_t std_slot(uint32_t c, int hb) { return (c * 0x9E3779B1u) >> (32 - hb); }

template <bool BF16>
__global__ __launch_bounds__(kStdThreads) void std_sample_kernel(DevPlan P, const void* x, int64_t T, int m,
                                                                 const int32_t* idx, StdWs W)
{
    extern __shared__ __align__(16) unsigned char smem[];
    const int js = blockIdx.x, l = blockIdx.y + 1, nb = blockIdx.z;
    const int Kp = P.active[l - 1], Dl = P.delta[l], n = Kp * Dl, d = P.d;
    if (16 * nb >= Kp) return;   // the level has fewer parent blocks (uniform per workgroup)
    const int64_t t = ((int64_t)js * T) / m;
    const int32_t* par = idx + t * P.k_tot + P.slot_base[l - 1];
    const uint32_t* g = P.gens + P.gens_off[l];
    int cbase = 0;
    for (int ll = 1; ll < l; ++ll) cbase += P.active[ll - 1] * P.delta[ll];
    StdRec* rec = W.rec + (int64_t)js * std_cands(P) + cbase;

    const int hb = std_hash_bits(P);
    const uint32_t hmask = (1u << hb) - 1u;
    int32_t* tab = (int32_t*)smem;   // candidate position e of the copy holding the slot, or -1
    unsigned char* rb = smem + align16u(4u << hb);
    uint32_t* pairs = (uint32_t*)rb;
    float* xf = (float*)rb;
    uint32_t* cw = (uint32_t*)(rb + align16u(BF16 ? P.prow * 4 : P.dp * 4));
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;

    for (int i = threadIdx.x; i < (1 << hb); i += kStdThreads) tab[i] = -1;
    if (wave == 0) {
        if constexpr (BF16) {
            load_pairs(P, lane, 1, 1, (const uint16_t*)x, t, pairs);
        } else {
            const float* xs = (const float*)x;
            for (int iota = lane; iota < P.dp; iota += 64) xf[iota] = iota < d ? xs[t * d + iota] : 0.f;
        }
    }
    {   // sign bitmaps of parents 16 nb .. 16 nb + 15: one nibble-table word per 4-bit group of the index
        const int col = threadIdx.x & 15, q = 16 * nb + col;
        const int32_t p = q < Kp ? par[q] : -1;
        const uint32_t pu = p >= 0 ? (uint32_t)p : 0u;
        for (int w = threadIdx.x >> 4; w < P.nchunk; w += kStdThreads / 16) {
            uint32_t word = 0;
            for (int gg = 0; gg < P.nt_groups; ++gg) word ^= P.nt[(gg * P.nchunk + w) * 16 + ((pu >> (4 * gg)) & 15u)];
            cw[col * P.cws + w] = p >= 0 ? word : 0u;
        }
    }
    __syncthreads();
    auto child = [&](int e) -> uint32_t {
        const int q = e / Dl;
        return (uint32_t)par[q] ^ g[e - q * Dl];
    };
    // every candidate of the level into the set (padding parents have none)
    for (int e = threadIdx.x; e < n; e += kStdThreads) {
        if (par[e / Dl] < 0) continue;
        const uint32_t c = child(e);
        uint32_t h = std_slot(c, hb);
        for (;;) {
            const int prev = atomicCAS(&tab[h], -1, e);
            if (prev == -1) break;   // inserted
            if (child(prev) == c) {  // the slot holds a copy: it keeps the lowest position
                atomicMin(&tab[h], e);
                break;
            }
            h = (h + 1u) & hmask;
        }
    }
    __syncthreads();

    const ActTile A{pairs, xf};
    const int col = lane & 15, kq = lane >> 4, q = 16 * nb + col;
    const int32_t p = q < Kp ? par[q] : -1;
    for (int mb = wave; mb < P.mblocks[l]; mb += kStdThreads / 64) {
        const f32x4 acc = mfma_scores<BF16>(P, lane, l, mb, 0, A, cw);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int jj = 16 * mb + 4 * kq + i;
            if (q >= Kp || jj >= Dl) continue;
            const int e = q * Dl + jj;
            StdRec r{-1, 0.f};
            if (p >= 0) {
                const uint32_t c = (uint32_t)p ^ g[jj];
                uint32_t h = std_slot(c, hb);
                int v = tab[h];
                while (v != e && v >= 0 && child(v) != c) {   // the child is in the set: the walk ends at its slot
                    h = (h + 1u) & hmask;
                    v = tab[h];
                }
                if (v == e) r = StdRec{(int32_t)c, acc[i] * P.rsd};
            }
            rec[e] = r;
        }
    }
}

__global__ void std_rec_clear_kernel(int64_t nrec, StdWs W)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nrec; i += (int64_t)gridDim.x * blockDim.x) {
        const StdRec r = W.rec[i];
        if (r.feat >= 0) W.acc[r.feat] = StdAcc{0u, 0xFFFFFFFFu, 0.0, 0.0};
    }
}

__global__ void std_rec_accum_kernel(int64_t nrec, StdWs W)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nrec; i += (int64_t)gridDim.x * blockDim.x) {
        const StdRec r = W.rec[i];
        if (r.feat < 0) continue;
        StdAcc* a = W.acc + r.feat;
        atomicAdd(&a->n, 1u);
        atomicAdd(&a->s1, (double)r.s);
        atomicAdd(&a->s2, (double)r.s * (double)r.s);
        atomicMin(&a->owner, (uint32_t)i);
    }
}

__global__ void std_rec_update_kernel(int64_t nrec, StdWs W, float2* stats, float* m2, float beta, float eps)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nrec; i += (int64_t)gridDim.x * blockDim.x) {
        const StdRec r = W.rec[i];
        if (r.feat < 0) continue;
        const StdAcc a = W.acc[r.feat];
        if (a.owner == (uint32_t)i) ema(stats, m2, r.feat, (double)a.n, a.s1, a.s2, beta, eps);
    }
}

dim3 std_grid(int64_t n, int threads)
{
    const int64_t need = (n + threads - 1) / threads;
    return dim3((unsigned)std::max<int64_t>(1, std::min<int64_t>(need, 4096)));
}

}  // namespace

bool std_supported(const DevPlan& P)
{
    for (int l = 1; l < P.levels; ++l)
        if (P.active[l - 1] * P.delta[l] > kStdMaxCand) return false;
    return P.d <= 16384 && std_sample_lds(P, false) <= (unsigned)kLdsBudget;
}

size_t std_workspace_bytes(const DevPlan& P)
{
    size_t total = 0;
    (void)std_ws(nullptr, P, &total);
    return total;
}

hipError_t launch_std_init(const DevPlan& P, float* stats, float* m2, hipStream_t stream)
{
    const int64_t N = (int64_t)1 << P.level_bits[P.levels - 1];
    hipLaunchKernelGGL(std_init_kernel, std_grid(N, 256), dim3(256), 0, stream, (float2*)stats, m2, N);
    return hipGetLastError();
}

hipError_t launch_std_update(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const int32_t* idx,
                             float beta, float eps, float* stats, float* m2, void* ws, hipStream_t stream)
{
    const StdWs W = std_ws(ws, P, nullptr);
    float2* st = (float2*)stats;
    const dim3 gc(kStdGroups, (P.d + 4 * kStdThreads - 1) / (4 * kStdThreads));
    const dim3 bc(kStdThreads * kStdColSlices);
    if (x_bf16) hipLaunchKernelGGL(std_col_kernel<true>, gc, bc, 0, stream, x, P.d, T, W);
    else hipLaunchKernelGGL(std_col_kernel<false>, gc, bc, 0, stream, x, P.d, T, W);
    hipLaunchKernelGGL(std_col_update_kernel, dim3((P.d + 255) / 256), dim3(256), 0, stream, P.d, T, W, st, m2, beta,
                       eps);
    const int m = (int)std::min<int64_t>(T, kStdSample);
    if (P.levels > 1 && m > 0) {
        const dim3 g2(m, P.levels - 1, std_parent_blocks(P));
        const size_t xl = std_sample_lds(P, x_bf16);
        if (x_bf16) {
            allow_lds(std_sample_kernel<true>, xl);
            hipLaunchKernelGGL(std_sample_kernel<true>, g2, dim3(kStdThreads), xl, stream, P, x, T, m, idx, W);
        } else {
            allow_lds(std_sample_kernel<false>, xl);
            hipLaunchKernelGGL(std_sample_kernel<false>, g2, dim3(kStdThreads), xl, stream, P, x, T, m, idx, W);
        }
        const int64_t nrec = (int64_t)m * std_cands(P);
        hipLaunchKernelGGL(std_rec_clear_kernel, std_grid(nrec, 256), dim3(256), 0, stream, nrec, W);
        hipLaunchKernelGGL(std_rec_accum_kernel, std_grid(nrec, 256), dim3(256), 0, stream, nrec, W);
        hipLaunchKernelGGL(std_rec_update_kernel, std_grid(nrec, 256), dim3(256), 0, stream, nrec, W, st, m2, beta,
                           eps);
    }
    return hipGetLastError();
}

}  // namespace dpb
