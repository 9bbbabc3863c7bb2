// Internal types shared by the host API and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <vector>

#include "tables.hpp"

namespace dpb {

constexpr int kMaxLevels = 8;
constexpr int kBlock = 256;               // threads per workgroup (4 wave64)
constexpr int kChunk = 32;                // coordinates per MFMA K step
constexpr int kLdsBudget = 160 * 1024;    // bytes of LDS a workgroup may use (gfx950: 160 KB per CU)

// Everything a kernel needs to know about a plan, passed by value.
struct DevPlan {
    int d;             // residual width
    int dp;            // d rounded up to a multiple of kChunk
    int nchunk;        // dp / kChunk
    int levels;
    int k_tot;
    int kmax;          // max_l K_l
    float rsd;         // fp32 round-to-nearest of 1/sqrt(d)
    int level_bits[kMaxLevels];
    int delta[kMaxLevels];      // Delta_l (0 for level 0)
    int active[kMaxLevels];     // K_l
    int slot_base[kMaxLevels];  // first code slot of level l
    int mblocks[kMaxLevels];    // ceil(Delta_l / 16)
    int cpad[kMaxLevels];       // K_{l-1} * Delta_l rounded up to a power of two
    int gens_off[kMaxLevels];   // offset of level l's generators in `gens`
    int64_t gamma_off[kMaxLevels];  // offset (in 16-byte units) of level l's A fragments
    const uint32_t* masks;      // [dp] row masks, zero past d
    const uint32_t* gens;       // generators, level by level
    const void* gamma;          // per level: [mblocks][nchunk][64 lanes] x 8 bf16 (+1/-1/0)

    // Code kernels (decode, decode-backward) and the scoring primitive.
    int wave_tokens;            // tokens a wave processes together (16 / cpt of the last level)
    int leaf_columns;           // 1: the last level decodes through parent columns on the matrix cores
    int cpt[kMaxLevels];        // parent columns per token at level l: K_{l-1} rounded up to a power of two
    int dpad[kMaxLevels];       // Delta_l rounded up to a multiple of 16
    int nt_groups;              // 4-bit index groups of the widest index
    int cws;                    // row stride of column bitmaps in LDS (odd, >= nchunk)
    int prow;                   // row stride (dwords) of bf16 activation pairs in LDS: dp/2 + 16
    int cpt_shift[kMaxLevels];  // log2 cpt[l]
    const uint32_t* nt;         // [max(nt_groups, kNtGroupsPadded)][nchunk][16] sign-bitmap word w of (v << 4g)
    int fr_cap;                 // slots per table-decode chunk (multiple of 32, <= kFrMax)
    int pb_bytes;               // bytes per coordinate of the leaf parents' sign bits (1 or 2)
    // Scoring A fragments in the interleaved-halves coordinate order: lane L,
    // element e = 2i + h of chunk c holds generator row 16*mb + L%16 at
    // coordinate 32c + 4*(L/16) + i + 16h.  Per level: [mblocks][nchunk][64] x 8 bf16.
    const void* gamma_pair;
    // Column-decode B fragments: lane L of block (cb, kb) holds generator rows
    // 16kb + 4*(L/16) + i (i < 4) at coordinate 16cb + L%16.  Per level:
    // [dp/16][dpad/16][64] x 4 bf16.
    const void* gamma_t;
    int64_t gamma_t_off[kMaxLevels];  // in 8-byte units
    // Collision-free hash of each level's generators: entry
    // h(x) = (x ^ (x >> gtab_shift[l])) & (2^gtab_bits[l] - 1) holds the pair
    // (g_j, j) of the generator with that hash, or (0, -1).
    const uint32_t* gtab;
    int gtab_off[kMaxLevels];   // in entries (pairs)
    int gtab_bits[kMaxLevels];
    int gtab_shift[kMaxLevels];
    int gtab_total;             // entries over all levels (0: routing disabled)
    int gens_total;             // sum_l Delta_l
    // Generator sign bitmaps: word (j, c) of level l at gbits_off[l] + j * cws + c
    // has bit b = sign of phi~_{g_j} at coordinate 32c + b (1: negative), for
    // j < gpad[l] = Delta_l rounded up to 32 (rows past Delta_l are zero; the
    // row stride cws = nchunk | 1 is the LDS layout, so a level is one copy).
    const uint32_t* gbits;
    int64_t gbits_off[kMaxLevels];
    int gpad[kMaxLevels];
    // 1: the backward takes <phi_s, g> of every slot directly instead of
    // scoring all children of each parent column (many children per parent)
    int bwd_direct;
};


// Per-wave LDS layout of the code kernels (byte offsets inside a wave's region).
struct CodeLayout {
    unsigned idx, coef, route, par, alpha, claim, fri, frc, frv, frt, pb, y, pairs, cw, score, bytes;
};

constexpr int kNtGroupsPadded = 8;   // nibble-table groups present on the device (zero words past nt_groups)
constexpr int kFrMax = 256;          // largest table-decode chunk
constexpr int kClaimed = 1 << 29;    // route flag: the slot is decoded through its column

__host__ __device__ inline unsigned align16u(unsigned v) { return (v + 15u) & ~15u; }

// The scoring buffers live inside the region of the output accumulator `y`,
// which is written only after scoring is done.  With fp32 activations the
// region holds the fp32 values instead of bf16 pairs, and the column bitmaps
// and scores follow it.
__host__ __device__ inline CodeLayout code_layout(const DevPlan& P, bool with_scoring, bool act_bf16 = true)
{
    CodeLayout L;
    const int TPW = P.wave_tokens, k = P.k_tot;
    const int dleaf = P.leaf_columns ? P.dpad[P.levels - 1] : 1;  // column coefficients of the last level
    unsigned off = 0;
    L.idx = off;   off = align16u(off + TPW * k * 4);
    L.coef = off;  off = align16u(off + TPW * k * 4);
    L.route = off; off = align16u(off + TPW * k * 4);
    L.par = off;   off = align16u(off + 16 * 4);
    L.fri = off;   off = align16u(off + P.fr_cap * 4);
    L.frc = off;   off = align16u(off + P.fr_cap * 4);
    L.frv = off = (off + 255u) & ~255u;  off += (P.fr_cap / 32) * 8 * 16 * 4;
    L.frt = off;   off = align16u(off + (P.fr_cap / 4) * 16 * 4);
    L.pb = off;    off = align16u(off + (P.leaf_columns ? TPW * P.dp * P.pb_bytes : 0));
    L.y = off;
    // column coefficients and claims are done with before y is written
    L.alpha = off;
    L.claim = align16u(off + 16 * dleaf * 4);
    unsigned yend = align16u(off + TPW * P.dp * 4);
    const unsigned cend = align16u(L.claim + 16 * dleaf * 4);
    if (cend > yend) yend = cend;
    L.pairs = L.cw = L.score = yend;
    off = yend;
    if (with_scoring) {
        unsigned s = act_bf16 ? L.y : yend;
        if (act_bf16) {
            L.pairs = s; s = align16u(s + TPW * P.prow * 4);
        } else {
            L.pairs = L.y;  // fp32 activations occupy the y region
        }
        L.cw = s;    s = align16u(s + 16 * P.cws * 4);
        L.score = s; s = align16u(s + 16 * 16 * 4);  // one 16 x 16 score tile
        off = s > yend ? s : yend;
    }
    L.bytes = (off + 255u) & ~255u;  // keeps every wave's table region 256-byte aligned
    return L;
}

constexpr int kCodeWaves = 4;  // waves per workgroup in the code kernels

// Shared (per-workgroup) LDS of the code kernels: row masks, generator hash
// tables and generators.  (The nibble tables are read through the cache.)
__host__ __device__ inline unsigned code_shared_bytes(const DevPlan& P)
{
    const unsigned b = align16u(P.dp * 4) + align16u(P.gtab_total * 8) + align16u(P.gens_total * 4);
    return (b + 255u) & ~255u;
}

// LDS layout of one encoder workgroup (byte offsets), shared by host and device.
struct EncodeLayout {
    int tile_tokens;    // tokens per workgroup
    int cpad_max;       // max_l cpad[l]
    unsigned off_x, off_par, off_key, bytes;
};

__host__ __device__ inline EncodeLayout encode_layout(const DevPlan& P, int x_bytes, int tile_tokens)
{
    EncodeLayout L;
    L.tile_tokens = tile_tokens;
    L.cpad_max = 1;
    for (int l = 1; l < P.levels; ++l)
        if (P.cpad[l] > L.cpad_max) L.cpad_max = P.cpad[l];
    unsigned off = (unsigned)P.dp * 4u;                     // row masks
    L.off_x = off;
    off += (unsigned)(tile_tokens * P.dp * x_bytes);        // activation tile
    L.off_par = off;
    off += (unsigned)(tile_tokens * P.kmax * 4);            // active parents
    off = (off + 15u) & ~15u;
    L.off_key = off;
    off += (unsigned)(tile_tokens * L.cpad_max * 8);        // candidate keys
    L.bytes = off;
    return L;
}

// Lets a kernel launch with more than 64 KB of dynamic LDS.
template <typename F>
inline void allow_lds(F* kernel, size_t bytes)
{
    if (bytes > 64 * 1024)
        (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

// True when the general encoder's workgroup (one fp32 token) fits the LDS budget.
bool general_encoder_fits(const DevPlan& P);

hipError_t launch_decode2(const DevPlan& P, const int32_t* idx, const float* coef, int64_t T, void* y,
                          bool y_bf16, hipStream_t stream);
hipError_t launch_decode_bwd2(const DevPlan& P, const int32_t* idx, const void* g, bool g_bf16, int64_t T,
                              float* grad_coef, void* grad_x, bool gx_bf16, hipStream_t stream,
                              const float* add_grad_coef = nullptr, const void* add_grad_x = nullptr,
                              const float* stats = nullptr);
bool code_kernels_fit(const DevPlan& P);
bool encode2_supported(const DevPlan& P);
bool encode2_std_supported(const DevPlan& P);
// Wide encoder (many children per parent): GEMM + selection per level.
bool encode_wide_supported(const DevPlan& P, bool x_bf16);
size_t encode_wide_workspace_bytes(const DevPlan& P, int64_t T);
// chunk: tokens per pass (0: the default, 16384), which sizes the workspace.
hipError_t launch_encode_wide(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const float* stats,
                              int32_t* idx, float* coef, void* ws, hipStream_t stream, int64_t chunk = 0);
// The allocation-free encoder's scratch (a device array of this size on each
// device): its address on `device`, which must be current (looked up once per
// device; nullptr on failure), and the tokens per pass it holds for a plan
// (0 if not even kStaticMinChunk tokens fit).
constexpr size_t kStaticScratchBytes = (size_t)64 << 20;
constexpr int64_t kStaticMinChunk = 256;
void* scratch_setup(int device);
int64_t static_chunk_tokens(const DevPlan& P);
hipError_t launch_encode2(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const float* stats, int32_t* idx,
                          float* coef, hipStream_t stream);

// EMA statistics of the score standardization (standardize.hip): tokens per
// batch on which the candidate moments of levels >= 1 are taken.
constexpr int kStdSample = 64;
size_t std_workspace_bytes(const DevPlan& P);
bool std_supported(const DevPlan& P);
hipError_t launch_std_init(const DevPlan& P, float* stats, float* m2, hipStream_t stream);
hipError_t launch_std_update(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const int32_t* idx,
                             float beta, float eps, float* stats, float* m2, void* ws, hipStream_t stream);

// Row epilogues, code edits and the variance loss (extras.hip).
hipError_t launch_normalize(int d, int64_t T, const void* u, bool u16, const void* ref, bool r16,
                            const int32_t* ref_rows, int64_t T_ref, void* y, bool y16, float* norms,
                            hipStream_t stream);
hipError_t launch_normalize_bwd(int d, int64_t T, const void* g, bool g16, const void* u, bool u16, const void* ref,
                                bool r16, void* gu, bool gu16, void* gr, bool gr16, int accumulate,
                                hipStream_t stream);
hipError_t launch_edit_codes(const int32_t* idx, const float* coef, const int32_t* tidx, const float* tcoef,
                             int64_t T, int k, const int32_t* rows, const int32_t* slots, const int32_t* ops,
                             int64_t E, int32_t* out_idx, float* out_coef, hipStream_t stream);
int variance_small_range(const int* level_bits, int levels);
bool variance_supported(int64_t nfeat, int S, int64_t nslots);
size_t variance_workspace_bytes(int64_t nfeat, int S, int64_t nslots);
hipError_t launch_variance_loss(const int32_t* idx, const float* coef, int64_t T, int k, int64_t nfeat, int S,
                                int n_min, void* ws, float* loss, float* grad, const float* grad_scale,
                                hipStream_t stream);
hipError_t launch_variance_grad(int64_t T, int k, int64_t nfeat, int S, void* ws, float* grad,
                                const float* grad_scale, hipStream_t stream);

// General encoder (encode_general.hip) for plans outside the narrow and wide encoders.
hipError_t launch_encode(const DevPlan& P, const void* x, bool x_bf16, int64_t T, const float* stats, int32_t* idx,
                         float* coef, hipStream_t stream);

}  // namespace dpb

struct dpb_plan {
    int device = -1;
    dpb::Hierarchy h;
    std::vector<uint32_t> masks_h;   // [d]
    std::vector<uint32_t> gens_h;    // sum Delta_l
    dpb::DevPlan dev{};
    void* dev_alloc = nullptr;       // one device allocation holding every table
};
