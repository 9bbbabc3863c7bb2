/*
 * dpb.h -- C ABI of the MI355X Deep Parity Bottleneck library (libdpb.so).
 *
 * The Deep Parity Bottleneck (DPB) of "Scaling Interpretable Transformers with
 * Parity Bottleneck Layers" maps a dense activation x in R^d to a sparse code
 * over N = 2^n features and back (§2, first paragraph).  Feature i < d is the
 * basis vector e_i; every other feature is the sign vector
 *     phi_i[iota] = (-1)^{popcount(M_iota & i) mod 2} / sqrt(d)
 * generated on chip from a small seed matrix M (§2.1 Eqs. 1-2; App. A.4,
 * packed-parity equation).  Features are arranged in levels; level l holds
 * the indices in [2^{n_{l-1}}, 2^{n_l}) (level 0: [0, d)), and the children of
 * a parent p are p XOR g_j for the level's generators g_j (§2.2).
 *
 * Conventions shared by every entry point
 *  - Token data (x, codes, y, gradients) are HIP DEVICE pointers owned by the
 *    caller, contiguous and row-major: activations [T, d], codes [T, k_tot].
 *    They must be 16-byte aligned.  The library never frees or retains them.
 *  - A code holds k_tot = sum_l K_l slots per token, level-major (the K_0 level-0
 *    slots first); within a level, slots are ordered by |coef| descending,
 *    then index ascending.  idx is the feature index (int32); coef its fp32
 *    coefficient.  The slot (idx = -1, coef = 0) is padding and is ignored.
 *  - `stream` is a hipStream_t (passed as void*; NULL = the default stream).
 *    Every compute call only enqueues work on it and returns; none
 *    allocates or synchronises.  The plan's tables live on the device that
 *    was current when the plan was created; calls must target that device.
 *  - Errors: argument errors are detected on the host before anything is
 *    enqueued and return a negative dpb_status; a failed launch returns
 *    DPB_EHIP (the HIP error is cleared).  No C++ exception crosses the ABI.
 *    T = 0 is a valid no-op.
 *  - Readings of points the paper leaves open are fixed by the library and
 *    listed in the repository's design notes: 0-based indices, bit p of an
 *    index pairs with column p of M, the modulus rule for p(z), the rows for d
 *    not a power of two, extra columns for n > 2t, and generator sampling.
 */
#ifndef DPB_H
#define DPB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DPB_MAX_LEVELS 8

typedef enum { DPB_F32 = 0, DPB_BF16 = 1 } dpb_dtype;

typedef enum {
    DPB_OK = 0,
    DPB_EINVAL = -1,       /* bad argument (shape, pointer, alignment, dtype) */
    DPB_EUNSUPPORTED = -2, /* valid per the paper but outside what this build supports */
    DPB_EHIP = -3,         /* a HIP runtime call or kernel launch failed */
    DPB_ENOMEM = -4        /* device or host allocation failed (plan creation only) */
} dpb_status;

/* Opaque plan: the hierarchy and the constant tables derived from it
 * (row masks M, generators, per-level child patterns).  Owns only those
 * KB-sized device tables. */
typedef struct dpb_plan dpb_plan;

const char* dpb_status_string(dpb_status s);

/* Per-level table (n_l, Delta_l, K_l) of App. G Table 6 from configuration
 * terms: `levels` counts level 0; n_0 = ceil(log2 d), n_{levels-1} = n_bits
 * and the levels in between are evenly spaced (rounded down); Delta_l =
 * branching for l >= 1 (Delta_0 = 0); K_l = beam below the last level and k
 * on the last.  Host only.  Outputs are arrays of `levels` ints. */
dpb_status dpb_hierarchy(int d, int n_bits, int levels, int branching, int beam, int k,
                         int* level_bits, int* branching_out, int* active_out);

/* Host-only construction of the plan's constant tables, for inspection:
 * masks_out[d] receives the packed rows M_iota (App. A.4, parity-mask-row
 * equation; bit q = column q), gens_out[sum_{l>=1} branching[l]] the
 * generators level by level (§2.2).  Touches no GPU. */
dpb_status dpb_build_tables(int d, int levels, const int* level_bits, const int* branching,
                            uint64_t seed, uint32_t* masks_out, uint32_t* gens_out);

/* Creates a plan from configuration terms (see dpb_hierarchy); `seed` selects
 * the generators.  Allocates the device tables on the current device. */
dpb_status dpb_plan_create(dpb_plan** out, int d, int n_bits, int levels, int branching,
                           int beam, int k, uint64_t seed);

/* Creates a plan from explicit per-level arrays of length `levels`:
 * level_bits[l] = n_l (n_0 >= ceil(log2 d), strictly increasing, n_last <= 30),
 * branching[l] = Delta_l (index 0 ignored), active[l] = K_l with
 * 1 <= K_0 <= d and 1 <= K_l <= K_{l-1} * Delta_l.  `generators` (host
 * pointer, may be NULL) supplies sum_{l>=1} Delta_l distinct generators, level
 * by level, each in [2^{n_{l-1}}, 2^{n_l}); NULL draws them from `seed`. */
dpb_status dpb_plan_create_ex(dpb_plan** out, int d, int levels, const int* level_bits,
                              const int* branching, const int* active,
                              const uint32_t* generators, uint64_t seed);

void dpb_plan_destroy(dpb_plan* plan);

/* k_tot = sum_l K_l, the slots per token of a code; 0 for a NULL plan. */
int dpb_plan_code_width(const dpb_plan* plan);

/* Copies the plan's hierarchy and host copies of its tables (any output may
 * be NULL): level_bits/branching/active [levels], masks [d], gens [sum Delta]. */
dpb_status dpb_plan_describe(const dpb_plan* plan, int* d, int* levels, int* level_bits,
                             int* branching, int* active, uint32_t* masks, uint32_t* gens);

/* ENCODE (§2.2): top-down beam search.  Level 0 scores every basis feature by
 * the coordinate itself (§2.1 Eq. 2) and keeps the K_0 of largest |x_iota|.
 * Each later level scores every child p XOR g_j of every active parent p,
 * s_c = <phi_c, x> = <gamma_j, phi~_p (.) x> (§2.2 child-scoring equation),
 * counts a child reached from several parents once, and keeps the K_l of
 * largest |s_c| (AbsTopK; ties to the lower index); coef = signed s_c.
 *   x    : device [T, d], fp32 or bf16 (x_dtype)
 *   idx  : device [T, k_tot] int32 (written)
 *   coef : device [T, k_tot] fp32  (written)
 * Scores accumulate in fp32; 1/sqrt(d) is applied once, after accumulation. */
dpb_status dpb_encode(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T,
                      int32_t* idx, float* coef, void* stream);

/* DECODE (§2.1): y = sum_slots coef * phi_idx, directions generated on chip.
 *   idx, coef : device [T, k_tot] (read; any valid code, not only encoder output)
 *   y         : device [T, d], fp32 or bf16 (y_dtype; written)
 * fp32 accumulation; bf16 output rounds to nearest even. */
dpb_status dpb_decode(const dpb_plan* plan, const int32_t* idx, const float* coef, int64_t T,
                      void* y, dpb_dtype y_dtype, void* stream);

/* DECODE BACKWARD: for upstream gradient g of y,
 *   grad_coef[s] = <phi_{idx_s}, g>                (the VJP of decode in coef)
 *   grad_x       = sum_s grad_coef[s] * phi_{idx_s} (through coef = Phi_S x,
 *                                                    indices held fixed)
 *   idx       : device [T, k_tot] int32 (read)
 *   grad_y    : device [T, d], fp32 or bf16 (g_dtype; read)
 *   grad_coef : device [T, k_tot] fp32 (written; 0 on padding slots)
 *   grad_x    : device [T, d], fp32 or bf16 (gx_dtype; written) */
dpb_status dpb_decode_bwd(const dpb_plan* plan, const int32_t* idx, const void* grad_y,
                          dpb_dtype g_dtype, int64_t T, float* grad_coef, void* grad_x,
                          dpb_dtype gx_dtype, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DPB_H */
