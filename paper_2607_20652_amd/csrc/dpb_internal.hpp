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
constexpr int kLdsBudget = 64 * 1024;     // bytes of LDS a workgroup may use

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
};

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

// True when every kernel's workgroup fits the LDS budget for this plan.
bool plan_fits(const DevPlan& P);

hipError_t launch_encode(const DevPlan& P, const void* x, bool x_bf16, int64_t T, int32_t* idx,
                         float* coef, hipStream_t stream);
hipError_t launch_decode(const DevPlan& P, const int32_t* idx, const float* coef, int64_t T, void* y,
                         bool y_bf16, hipStream_t stream);
hipError_t launch_decode_bwd(const DevPlan& P, const int32_t* idx, const void* g, bool g_bf16, int64_t T,
                             float* grad_coef, void* grad_x, bool gx_bf16, hipStream_t stream);

}  // namespace dpb

struct dpb_plan {
    int device = -1;
    dpb::Hierarchy h;
    std::vector<uint32_t> masks_h;   // [d]
    std::vector<uint32_t> gens_h;    // sum Delta_l
    dpb::DevPlan dev{};
    void* dev_alloc = nullptr;       // one device allocation holding every table
};
