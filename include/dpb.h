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
    DPB_EUNSUPPORTED = -2, /* valid per the paper but outside what this library supports */
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
 * by level, each in [2^{n_{l-1}}, 2^{n_l}); NULL draws them from `seed`.
 * DPB_EINVAL for arrays that break these rules.  DPB_EUNSUPPORTED for valid
 * plans outside the library's limits: d > 4096; n_last > 3t or 2t > 31 with
 * t = ceil(log2 d) (the mask construction of App. A.4 over GF(2^t)); any
 * K_l > 256; any Delta_l > 4096 or K_{l-1} Delta_l > 8192 candidates per
 * token and level; sum_l K_l > 1024; and plans whose one-token encoder or
 * one-token decode rows exceed the 160 KB of LDS of a compute unit. */
dpb_status dpb_plan_create_ex(dpb_plan** out, int d, int levels, const int* level_bits,
                              const int* branching, const int* active,
                              const uint32_t* generators, uint64_t seed);

void dpb_plan_destroy(dpb_plan* plan);

/* k_tot = sum_l K_l, the slots per token of a code; 0 for a NULL plan. */
int dpb_plan_code_width(const dpb_plan* plan);

/* Host copies of the plan's constant tables, for checking them against an
 * independent construction: masks_host [d] receives the packed rows M_iota
 * (App. A.4, parity-mask-row equation; bit q = column q), gens_host
 * [sum_{l>=1} Delta_l] the generators level by level (§2.2).  Host pointers
 * owned by the caller; gens_host may be NULL for a one-level plan.  Touches
 * no GPU.  DPB_EINVAL for a NULL plan or a missing output. */
dpb_status dpb_plan_tables(const dpb_plan* plan, uint32_t* masks_host, uint32_t* gens_host);

/* Copies the plan's hierarchy and host copies of its tables (any output may
 * be NULL): level_bits/branching/active [levels], masks [d], gens [sum Delta]. */
dpb_status dpb_plan_describe(const dpb_plan* plan, int* d, int* levels, int* level_bits,
                             int* branching, int* active, uint32_t* masks, uint32_t* gens);

/* Bytes of device workspace dpb_encode and dpb_encode_std need for T
 * tokens (the same for either activation type, with or without statistics;
 * 0 for a NULL plan or T <= 0).  0 when the plan runs on the narrow encoder
 * (at most 64 children per parent, K_0 up to the lanes a token gets, and the
 * other limits of that kernel) or on the general one; for plans that score
 * many children per parent (up to 256, as the paper's own hierarchies do,
 * App. G Table 6), for up to C = min(T, 16384) tokens per pass, a region of
 * 4 * max_l K_{l-1} Delta_l bytes per token (it holds the token's listed
 * candidates, or all its child scores) and one 4-byte count per token, each
 * part rounded up to 256 bytes (512 MiB for the paper's 3-level hierarchy at
 * 16384 tokens). */
size_t dpb_encode_workspace_bytes(const dpb_plan* plan, int64_t T);

/* ENCODE (§2.2): top-down beam search.  Level 0 scores every basis feature by
 * the coordinate itself (§2.1 Eq. 2) and keeps the K_0 of largest |x_iota|.
 * Each later level scores every child p XOR g_j of every active parent p,
 * s_c = <phi_c, x> = <gamma_j, phi~_p (.) x> (§2.2 child-scoring equation),
 * counts a child reached from several parents once, and keeps the K_l of
 * largest |s_c| (AbsTopK; ties to the lower index); coef = signed s_c.
 *   x         : device [T, d], fp32 or bf16 (x_dtype)
 *   idx       : device [T, k_tot] int32 (written)
 *   coef      : device [T, k_tot] fp32  (written)
 *   workspace : device scratch of ws_bytes bytes, caller-owned, 16-B aligned,
 *               overwritten (nothing needs clearing); may be NULL when
 *               dpb_encode_workspace_bytes(plan, T) is 0.  A plan that needs
 *               one and is given none, or too little, gets DPB_EINVAL before
 *               anything is enqueued.
 * Scores accumulate in fp32; 1/sqrt(d) is applied once, after accumulation.
 * Plans with many children per parent run each level as a matrix-core GEMM
 * of all K_{l-1} x Delta_l child scores whose epilogue lists each token's
 * candidates above a threshold in the workspace, followed by the AbsTopK
 * selection; the results are those of the definition either way. */
dpb_status dpb_encode(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, int32_t* idx,
                      float* coef, void* workspace, size_t ws_bytes, void* stream);

/* DECODE (§2.1): y = sum_slots coef * phi_idx, directions generated on chip.
 *   idx, coef : device [T, k_tot] (read; any valid code, not only encoder output)
 *   y         : device [T, d], fp32 or bf16 (y_dtype; written)
 * fp32 accumulation; bf16 output rounds to nearest even. */
dpb_status dpb_decode(const dpb_plan* plan, const int32_t* idx, const float* coef, int64_t T,
                      void* y, dpb_dtype y_dtype, void* stream);

/* FORWARD: dpb_encode (stats NULL) or dpb_encode_std (stats given) followed
 * by dpb_decode of the code just written (§2.2 beam search, then §2.1 Eq. 1),
 * in one call; idx, coef and y are those calls' results bit for bit:
 *   x, stats, idx, coef, workspace, ws_bytes : as in dpb_encode / dpb_encode_std
 *                                              (the same workspace rule)
 *   y         : device [T, d], fp32 or bf16 (y_dtype; written), 16-B aligned
 * The encoder and the decode kernel are enqueued in turn on `stream`.  Errors
 * as dpb_encode's, plus DPB_EINVAL for a NULL or misaligned y or an unknown
 * y_dtype, found before anything is enqueued. */
dpb_status dpb_forward(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const float* stats,
                       int32_t* idx, float* coef, void* y, dpb_dtype y_dtype, void* workspace, size_t ws_bytes,
                       void* stream);

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

/* DECODE BACKWARD with extra gradient terms, for a layer whose loss also
 * depends on the coefficients directly (the variance auxiliary loss of §2.2,
 * "Auxillary losses") and on the bottleneck input through a path other than
 * the code (the norm of the normalized reconstruction, §2.2 "Normalized
 * Reconstruction"):
 *   grad_coef[s] = <phi_{idx_s}, g> + add_grad_coef[s]
 *   grad_x       = sum_s grad_coef[s] * phi_{idx_s} + add_grad_x
 *   add_grad_coef : device [T, k_tot] fp32, or NULL for none (read)
 *   add_grad_x    : device [T, d] in gx_dtype, or NULL for none (read); may
 *                   be the same buffer as grad_x (each element is read
 *                   before it is written, by the same thread).
 *   stats         : the standardization statistics the code was encoded
 *                   with (see dpb_encode_std), or NULL.  A standardized
 *                   coefficient z = (s - mu) r moves with x as r phi, so
 *                   grad_x = sum_s grad_coef[s] r_{idx_s} phi_{idx_s} + add_grad_x
 *                   (grad_coef itself is unchanged).
 * Every other argument as in dpb_decode_bwd; with all three extras NULL the
 * results equal dpb_decode_bwd's. */
dpb_status dpb_decode_bwd_ex(const dpb_plan* plan, const int32_t* idx, const void* grad_y,
                             dpb_dtype g_dtype, int64_t T, const float* add_grad_coef,
                             const void* add_grad_x, const float* stats, float* grad_coef,
                             void* grad_x, dpb_dtype gx_dtype, void* stream);

/* ENCODE WITHOUT ALLOCATION, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the results of dpb_encode (stats NULL) or of dpb_encode_std
 * (stats given), bit for bit, without a caller workspace.  Plans that need
 * one (dpb_encode_workspace_bytes > 0) take it from a scratch array the
 * library holds on each device it runs on, DPB_NOALLOC_SCRATCH_BYTES bytes,
 * kept until the process ends, and go through the tokens in passes sized to
 * it, so any T is accepted; a plan for which a pass of 256 tokens would not
 * fit gets DPB_EUNSUPPORTED (none of the plans the library accepts).  The
 * array's device address is looked up when a plan is created on the device.
 * Every call on one GPU uses that GPU's array: calls that may overlap in
 * time on one GPU (other streams or threads) race and must be serialized by
 * the caller.  Nothing in the array needs to start cleared.  Allocates and
 * frees nothing.  Other arguments as dpb_encode / dpb_encode_std. */
#define DPB_NOALLOC_SCRATCH_BYTES (64u << 20)

dpb_status dpb_encode_noalloc(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T,
                              const float* stats, int32_t* idx, float* coef, void* stream);

/* SCORE STANDARDIZATION (§2.2 "Score Standardization").  The state is two
 * caller-owned device arrays over all N = 2^n_last features:
 *   stats : fp32 [N][2] = (mu, r): the moving average of the feature's raw
 *           score and r = 1 / sigma, sigma^2 = m2 - mu^2 + eps at the last update
 *   m2    : fp32 [N], the moving average of the squared raw score
 * Initial state (dpb_std_init): mu = 0, r = 1, m2 = 1 -- with it the
 * standardized encoder equals dpb_encode. */
#define DPB_STD_SAMPLE 64   /* tokens per batch for the moments of levels >= 1 */

dpb_status dpb_std_init(const dpb_plan* plan, float* stats, float* m2, void* stream);

/* ENCODE on standardized scores: every candidate's raw score s_c becomes
 * z_c = (s_c - mu_c) r_c; AbsTopK runs on |z| (ties to the lower index) and
 * z is the coefficient written to the code.  Level-0 z is computed in fp32
 * as (x - mu) * r.  Arguments as dpb_encode (the same workspace rule), plus
 *   stats : device fp32 [N][2] (read; required).
 * Every plan the library accepts is supported (each encoder has a
 * standardized form). */
dpb_status dpb_encode_std(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const float* stats,
                          int32_t* idx, float* coef, void* workspace, size_t ws_bytes, void* stream);

/* Bytes of device workspace dpb_std_update needs (0 for a NULL plan):
 * 32 bytes per feature, 4 KiB per coordinate, and 8 bytes per candidate of
 * the sampled tokens. */
size_t dpb_std_workspace_bytes(const dpb_plan* plan);

/* EMA UPDATE after a batch encoded with dpb_encode_std (x, T, and its code
 * idx).  Each feature's sample is its raw scores on the tokens where it was
 * a candidate: every token for a basis feature (s = x_iota); for a feature
 * of level l >= 1, the tokens t_j = floor(j T / m), j < m = min(T, 64), at
 * which it is a child p XOR g_j of an active parent p (a level l-1 entry of
 * that token's code), counted once per token, s = <phi_c, x_t>.  A feature
 * with samples s_1..s_n gets moving averages of its first two raw moments,
 *   mu <- (1 - momentum) mu + momentum mean(s),
 *   m2 <- (1 - momentum) m2 + momentum mean(s^2),
 *   r = 1 / sqrt(max(m2 - mu^2, 0) + eps)
 * (so a feature sampled once per batch still measures its spread across
 * batches); other features keep their state.  Sums of s and s^2 accumulate
 * in fp64, the state update is fp32.  Supported while every level's
 * K_{l-1} Delta_l is at most 8192 and d at most 16384 (else DPB_EUNSUPPORTED).
 *   momentum in [0, 1], eps >= 0
 *   stats, m2  : device (read and written)
 *   workspace  : device, >= dpb_std_workspace_bytes(plan), 16-B aligned;
 *                caller-owned scratch, overwritten, no clearing needed */
dpb_status dpb_std_update(const dpb_plan* plan, const void* x, dpb_dtype x_dtype, int64_t T, const int32_t* idx,
                          float momentum, float eps, float* stats, float* m2, void* workspace, size_t ws_bytes,
                          void* stream);

/* NORMALIZED RECONSTRUCTION (§2.2 "Normalized Reconstruction"): each row of
 * the decoder output u is rescaled to the norm of the bottleneck input,
 *   y_t = u_t * ||ref_{r(t)}|| / ||u_t||,   y_t = 0 where ||u_t|| = 0,
 * with r(t) = ref_rows[t] if ref_rows is given, else t (the greedy feature
 * editing of App. C.3 rescales edited codes to their source row's norm).
 *   u        : device [T, d], u_dtype (read)
 *   ref      : device [T_ref, d], ref_dtype (read)
 *   ref_rows : device [T] int32, or NULL (then T_ref must equal T); a row
 *              index outside [0, T_ref) counts as a reference of norm 0
 *   y        : device [T, d], y_dtype (written; may be the same buffer as u
 *              when u_dtype == y_dtype)
 *   norms    : device [T, 2] fp32 (||ref_{r(t)}||, ||u_t||), or NULL
 * Sums of squares accumulate in fp32.  d comes from the plan. */
dpb_status dpb_normalize(const dpb_plan* plan, const void* u, dpb_dtype u_dtype, const void* ref,
                         dpb_dtype ref_dtype, const int32_t* ref_rows, int64_t T_ref, int64_t T,
                         void* y, dpb_dtype y_dtype, float* norms, void* stream);

/* Backward of dpb_normalize (ref_rows = NULL) for upstream gradient g of y:
 *   grad_u   = (||ref|| / ||u||) (g - (<g,u> / ||u||^2) u)
 *   grad_ref = (<g,u> / (||u|| ||ref||)) ref        (added to grad_ref when
 *                                                    accumulate != 0)
 * both 0 where ||u|| = 0, and grad_ref = 0 where ||ref|| = 0.
 *   g, u, ref        : device [T, d] in their dtypes (read)
 *   grad_u, grad_ref : device [T, d] in their dtypes (written; must not
 *                      overlap each other or the inputs) */
dpb_status dpb_normalize_bwd(const dpb_plan* plan, const void* g, dpb_dtype g_dtype, const void* u,
                             dpb_dtype u_dtype, const void* ref, dpb_dtype ref_dtype, int64_t T,
                             void* grad_u, dpb_dtype gu_dtype, void* grad_ref, dpb_dtype gr_dtype,
                             int accumulate, void* stream);

/* Operations of the greedy feature editing of App. C.3 (fine-grained causal
 * intervention); each edits one slot position of a source code using a
 * target code. */
typedef enum {
    DPB_EDIT_ZERO = 0,    /* coefficient := 0 */
    DPB_EDIT_REPLACE = 1, /* index and coefficient := the target's at the same position */
    DPB_EDIT_RESCALE = 2, /* coefficient := the target's at the same position; index kept */
    DPB_EDIT_NONE = 3     /* unchanged copy of the source row */
} dpb_edit_op;

/* CODE EDITS: one output code per edit e, equal to source row rows[e] with
 * the slot at position slots[e] (a column of the level-major code) changed by
 * ops[e].  Slots at the same position belong to the same level, so a
 * replaced index stays in that level's index range.
 *   idx, coef         : device [T, k_tot] source code (read)
 *   tgt_idx, tgt_coef : device [T, k_tot] target code (read), or both NULL
 *                       (then only ZERO and NONE are valid)
 *   rows, slots, ops  : device [E] int32 (read)
 *   out_idx, out_coef : device [E, k_tot] (written; must not overlap the
 *                       inputs)
 * An edit whose row, slot or op is out of range (or needs the missing
 * target) yields an all-padding output row (idx -1, coef 0): edit lists live
 * on the device and are not inspected by the host. */
dpb_status dpb_edit_codes(const dpb_plan* plan, const int32_t* idx, const float* coef,
                          const int32_t* tgt_idx, const float* tgt_coef, int64_t T,
                          const int32_t* rows, const int32_t* slots, const int32_t* ops, int64_t E,
                          int32_t* out_idx, float* out_coef, void* stream);

/* Bytes of device workspace dpb_variance_loss needs for a batch of T tokens
 * (0 for a NULL plan or T < 0): 16 bytes per slot (T * k_tot), 2 KiB per
 * feature of the low levels (the S <= 4096 smallest indices, counted per
 * workgroup), and about 1 KiB per bucket of 1024 to 4096 other features;
 * each part 256-byte aligned.  About 105 MiB for 65536 tokens at N = 2^20,
 * k_tot = 96. */
size_t dpb_variance_workspace_bytes(const dpb_plan* plan, int64_t T);

/* VARIANCE AUXILIARY LOSS (§2.2 "Auxillary losses" equation) over a batch of
 * codes: the coefficients of the slots holding feature i form its sample;
 * F = features with at least n_min samples;
 *   loss = -(1/|F|) sum_{i in F} Var_i      (population variance; 0 if F is empty)
 *   grad_coef[s] = d loss / d coef[s] = -(2/|F|) (coef[s] - mean_i) / count_i
 *                  for slots of features in F, else 0.
 * Slots whose index is outside [0, N) (padding) are not samples.
 *   idx, coef  : device [T, k_tot] (read)
 *   workspace  : device, >= dpb_variance_workspace_bytes(plan, T) bytes,
 *                16-B aligned; caller-owned scratch, overwritten (nothing in it
 *                needs to be cleared); afterwards it holds what
 *                dpb_variance_grad reads
 *   loss       : device fp32 scalar (written)
 *   grad_coef  : device [T, k_tot] fp32 (written), or NULL for the loss only
 *   grad_scale : device fp32 scalar multiplying grad_coef (the upstream
 *                gradient of the loss in a backward pass), or NULL for 1
 * Features of the low levels accumulate sums, then squared deviations about
 * the mean, in fp32; the others sums of a and a^2 in fp64.  Both use LDS
 * atomics, whose order (and so the last bits) may vary from run to run; the
 * sum over features is taken in fp64 in a fixed order.  T = 0 still writes
 * loss = 0.  DPB_EUNSUPPORTED when N exceeds 2^24 + 4096 or T * k_tot
 * reaches 2^31. */
dpb_status dpb_variance_loss(const dpb_plan* plan, const int32_t* idx, const float* coef, int64_t T,
                             int n_min, void* workspace, size_t ws_bytes, float* loss, float* grad_coef,
                             const float* grad_scale, void* stream);

/* Gradient of the variance auxiliary loss alone (a backward pass after a
 * forward that computed the loss): from what a dpb_variance_loss call over T
 * tokens left in `workspace`, writes grad_coef [T, k_tot] exactly as that
 * call would have, times *grad_scale (NULL: 1).  The workspace must not have
 * been used by another call in between; it is only read. */
dpb_status dpb_variance_grad(const dpb_plan* plan, int64_t T, const void* workspace, size_t ws_bytes,
                             float* grad_coef, const float* grad_scale, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DPB_H */
