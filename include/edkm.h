/*
 * edkm.h — C ABI of the MI355X (gfx950) eDKM hot path: DKM weight clustering,
 * forward and backward, computed on the 16-bit uniquified attention table.
 *
 * The method (paper: "eDKM: An Efficient and Accurate Train-time Weight
 * Clustering for Large Language Models", Sec. 2 and 2.2):
 *
 *   DKM (Sec. 2) clusters a weight tensor W against k = 2^b centroids C through
 *   an attention map A_ij = softmax_j(-|w_i - c_j| / tau), iterates
 *   C_j = sum_i A_ij w_i / sum_i A_ij, and outputs W~ = A C; training needs
 *   the backward of W~ with respect to W and C.  The map is O(|W||C|).
 *
 *   Uniquification (Sec. 2.2, Fig. "mem_dkm:flow"): a 16-bit weight has at most
 *   65,536 distinct bit patterns and equal patterns have equal attention rows,
 *   so the map becomes an attention table with one row per pattern plus an
 *   index list whose entry is the weight's own pattern.  Here every sum over
 *   weights becomes a sum over table rows weighted by per-pattern counts, and
 *   the N-sized work reduces to a histogram, a keyed gradient sum and two
 *   gathers.  edkm_unique_inverse returns the compacted form of the two lists
 *   (sorted distinct patterns, each weight's position among them) for callers
 *   that store them; edkm_palettize exports the clustered result.
 *
 * Conventions for every entry point:
 *   - Weights are 16-bit floats, fp16 (IEEE binary16, the default) or bf16
 *     (bfloat16, the paper's training format, Sec. 3), chosen per plan and
 *     passed as their raw bit patterns (uint16_t), flat, any shape (all
 *     operations are elementwise in the weight index).  A pattern is a table
 *     key; +0 and -0 are distinct keys of equal value.
 *   - Device pointers are HIP device memory owned by the caller.  The library
 *     allocates nothing and keeps no global state; all calls are asynchronous
 *     on the given stream except where noted.  Pointers need only natural
 *     alignment (2 bytes for keys, 4 for floats); 16-byte-aligned buffers take
 *     the vectorised path.
 *   - Per-matrix state lives in two caller-owned places: an edkm_plan (host
 *     memory, filled by edkm_plan_init) and a device workspace of
 *     edkm_workspace_bytes() bytes.  Calls on one plan must be issued in the
 *     order init_unique -> forward -> backward (or forward_dense ->
 *     backward_dense) on one stream, with the same key buffer and unchanged
 *     keys; a call out of order returns EDKM_ERR_STATE before touching the
 *     GPU.  edkm_unique_inverse may follow init_unique at any point of that
 *     sequence; edkm_palettize needs no earlier call.  Distinct plans with
 *     distinct workspaces may be used concurrently.
 *   - Errors are returned, never thrown; argument errors are detected on the
 *     host before any HIP call and leave the plan unchanged.  After
 *     EDKM_ERR_HIP the workspace may hold a half-done step, so the plan falls
 *     back: a failed init_unique (or forward_dense) needs a new init_unique,
 *     a failed forward or backward a new forward.
 *   - Every entry point can be captured in a HIP graph (no allocation, no
 *     memset, no synchronisation), except init_unique with check_finite = 1,
 *     which synchronises.  A replay repeats the device work of the captured
 *     calls on the buffers they were given.
 */
#ifndef EDKM_H
#define EDKM_H

#include <stddef.h>
#include <stdint.h>
/* The HIP runtime header wants the platform named when a plain C or C++
 * compiler (not hipcc) includes it; this library exists for AMD GPUs only. */
#ifndef __HIP_PLATFORM_AMD__
#define __HIP_PLATFORM_AMD__ 1
#endif
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EDKM_NKEYS 65536        /* table rows: every 16-bit pattern */
#define EDKM_MAX_BITS 4         /* k = 2^bits <= 16 centroids */
#define EDKM_MAX_ITER 1024
#define EDKM_MAX_N 4294967295ull /* per matrix; counts are uint32 */
#define EDKM_LAUNCH_GROUP 28    /* matrices per launch in the batched forms (four decoder layers) */

typedef int edkm_status;
enum {
    EDKM_OK = 0,
    EDKM_ERR_ARG = -1,        /* invalid argument (null pointer, size, bits, tau, ...) */
    EDKM_ERR_NONFINITE = -2,  /* a weight is Inf or NaN (only reported when checked) */
    EDKM_ERR_WORKSPACE = -3,  /* workspace null, too small, or misaligned (256 B) */
    EDKM_ERR_STATE = -4,      /* call out of order for this plan, or different keys */
    EDKM_ERR_HIP = -5         /* a HIP runtime call failed */
};

/* Host-side per-matrix record.  Opaque; the caller owns the memory (stack or
 * heap) and must not copy it between calls: the record knows its own address,
 * and a copy is refused (EDKM_ERR_ARG) by every call but edkm_plan_init. */
typedef struct edkm_plan {
    uint64_t opaque[32];
} edkm_plan;

/* Device workspace size for one matrix of n weights with k = 2^bits
 * centroids and up to max_iter DKM iterations; 0 if the arguments are invalid.
 * It is about 40 MiB and does not grow with n. */
size_t edkm_workspace_bytes(uint64_t n, int bits, int max_iter);

/* Weight formats. */
enum {
    EDKM_KEYS_FP16 = 0,   /* IEEE 754 binary16 */
    EDKM_KEYS_BF16 = 1    /* bfloat16: the upper half of a binary32 */
};

/* Set up a plan for n (1..EDKM_MAX_N) fp16 weights, bits in 1..4, max_iter in
 * 1..EDKM_MAX_ITER, with ws a device buffer of ws_bytes >= the size above,
 * 256-byte aligned, used only by this plan.  Host only; no HIP call. */
edkm_status edkm_plan_init(edkm_plan* plan, uint64_t n, int bits, int max_iter,
                           void* ws, size_t ws_bytes);

/* edkm_plan_init for weights of the given format (EDKM_KEYS_FP16 or
 * EDKM_KEYS_BF16; anything else is EDKM_ERR_ARG).  The format decides how a
 * pattern decodes to its value, which patterns are Inf/NaN, and the type of
 * 16-bit W~ outputs.  Host only; no HIP call. */
edkm_status edkm_plan_init_ex(edkm_plan* plan, uint64_t n, int bits, int max_iter,
                              int key_format, void* ws, size_t ws_bytes);

/* Uniquification (Sec. 2.2): counts[u] = #{i : w_bits[i] = u} for all 65,536
 * patterns, kept in the workspace for forward/backward.
 *   w_bits         device, n patterns
 *   counts_out     nullable, device uint32[65536]: copy of the counts
 *   num_unique_out nullable, device uint32[1]: number of occupied patterns
 *   check_finite   1: synchronise the stream and return EDKM_ERR_NONFINITE if
 *                  any weight is Inf/NaN; 0: no sync, and non-finite weights are
 *                  left out of the clustering (their outputs are NaN).
 * The counts are exact (integer).  Cost: one read of the keys. */
edkm_status edkm_init_unique(edkm_plan* plan, const uint16_t* w_bits,
                             uint32_t* counts_out, uint32_t* num_unique_out,
                             int check_finite, hipStream_t stream);

/* DKM forward on the table (Sec. 2, Sec. 2.2).  For t = 1..T:
 *   a_uj = softmax_j(-|v_u - C^(t-1)_j| / tau) for each occupied pattern u
 *   (v_u its value), S_j = sum_u n_u a_uj, P_j = sum_u n_u a_uj v_u,
 *   C^(t)_j = P_j / S_j (a centroid with S_j = 0 keeps its value).
 * T = max_iter, or the first t with max_j |C^(t)_j - C^(t-1)_j| <= eps when
 * eps > 0.  Output W~_i = sum_j a^(T)_{w_i, j} C^(T)_j, i.e. a gather of the
 * table row of w_i's pattern.
 *   w_bits     device, n patterns; must be the buffer given to init_unique
 *   tau        > 0, finite;  eps >= 0 (0: exactly max_iter iterations)
 *   c_in       device float[k]: C^(0)
 *   c_out      device float[k]: C^(T)
 *   w_tilde    device, n outputs: float, or, if out_half = 1, 16-bit floats
 *              of the plan's weight format (fp16 or bf16 bits, uint16; round to
 *              nearest even)
 *   iters_out  nullable, device int32[1]: T
 * Arithmetic is fp32 with fixed-order reductions: results are bitwise
 * repeatable.  Saves C^(0..T), S^(1..T) and the table in the workspace. */
edkm_status edkm_forward(edkm_plan* plan, const uint16_t* w_bits, float tau, float eps,
                         const float* c_in, float* c_out, void* w_tilde, int out_half,
                         int32_t* iters_out, hipStream_t stream);

/* DKM backward (the gradient that autograd of the dense map gives, Sec. 2.2),
 * for L with dL/dW~ = grad_w_tilde, through all T iterations:
 *   G_u = sum_{i: w_bits[i] = u} grad_w_tilde[i]   (keyed reduction)
 *   dL/dw_i = grad_w_tilde[i] * H[w_bits[i]] + R[w_bits[i]]
 * with H, R and dL/dC^(0) from the analytic softmax Jacobian on the table.
 *   grad_w_tilde  device float[n]
 *   grad_w        device float[n]
 *   grad_c        device float[k]: dL/dC^(0)
 * d|x|/dx at x = 0 is 0.  The keyed reduction uses float atomics, so results
 * vary in the last bits between runs.  May be repeated after one forward (with
 * other gradients); after EDKM_ERR_HIP it needs a new forward first. */
edkm_status edkm_backward(edkm_plan* plan, const uint16_t* w_bits, const float* grad_w_tilde,
                          float* grad_w, float* grad_c, hipStream_t stream);

/* edkm_backward (the same gradient, Sec. 2.2) with 16-bit N-sized gradient
 * arrays, for training in the weights' own precision (the 16-bit W~ of
 * forward with out_half = 1 gets a 16-bit dL/dW~ from autograd, and dL/dw
 * goes back to fp16 or bf16 weights): flags is a bitwise or of
 *   EDKM_GRAD_IN_HALF   grad_w_tilde holds n 16-bit floats of the plan's
 *                       weight format (fp16 or bf16 bits, uint16), else float;
 *   EDKM_GRAD_OUT_HALF  grad_w receives n 16-bit floats of that format
 *                       (rounded to nearest even from the fp32 result), else
 *                       float.
 * Each halves the bytes its array moves (the keyed sum reads grad_w_tilde,
 * the gradient gather reads grad_w_tilde and writes grad_w).  The arithmetic
 * is the same fp32 as edkm_backward's; with both flags 0 it is edkm_backward.
 * Other flag bits are EDKM_ERR_ARG. */
enum { EDKM_GRAD_IN_HALF = 1, EDKM_GRAD_OUT_HALF = 2 };
edkm_status edkm_backward_ex(edkm_plan* plan, const uint16_t* w_bits, const void* grad_w_tilde,
                             void* grad_w, float* grad_c, int flags, hipStream_t stream);

/* Batched forms: `count` independent matrices (own plan, keys and outputs;
 * same tau and eps) processed together.  The batch is cut into launch groups
 * of up to EDKM_LAUNCH_GROUP consecutive matrices with the same bit width and
 * weight format, and each step of the path is one launch per group.  Arrays
 * are host arrays of `count` entries (count >= 1, any size: groups are formed
 * by the library); entries of the nullable output arrays may be NULL, and the
 * arrays themselves may be NULL.  Equivalent to calling the single-matrix
 * form on each (with check_finite = 1, a matrix with Inf/NaN weights leaves
 * only its own plan uncounted; the call then returns EDKM_ERR_NONFINITE). */
edkm_status edkm_init_unique_batch(int count, edkm_plan* const* plans,
                                   const uint16_t* const* w_bits,
                                   uint32_t* const* counts_out,
                                   uint32_t* const* num_unique_out,
                                   int check_finite, hipStream_t stream);
edkm_status edkm_forward_batch(int count, edkm_plan* const* plans,
                               const uint16_t* const* w_bits, float tau, float eps,
                               const float* const* c_in, float* const* c_out,
                               void* const* w_tilde, int out_half,
                               int32_t* const* iters_out, hipStream_t stream);
edkm_status edkm_backward_batch(int count, edkm_plan* const* plans,
                                const uint16_t* const* w_bits,
                                const float* const* grad_w_tilde,
                                float* const* grad_w, float* const* grad_c,
                                hipStream_t stream);
edkm_status edkm_backward_batch_ex(int count, edkm_plan* const* plans,
                                   const uint16_t* const* w_bits,
                                   const void* const* grad_w_tilde,
                                   void* const* grad_w, float* const* grad_c,
                                   int flags, hipStream_t stream);

/* Dense (non-uniquified) DKM for comparison (Sec. 2: the O(|W||C|) map):
 * the same mathematics evaluated per weight over the N x k map, recomputing
 * the map row of every weight in every pass.  Same arguments and outputs as
 * edkm_forward; needs no init_unique.  attn_out (nullable, device
 * float[n * k], row-major) receives the final map A^(T). */
edkm_status edkm_forward_dense(edkm_plan* plan, const uint16_t* w_bits, float tau, float eps,
                               const float* c_in, float* c_out, void* w_tilde, int out_half,
                               int32_t* iters_out, float* attn_out, hipStream_t stream);

/* Backward of edkm_forward_dense, same contract as edkm_backward
 * (deterministic: no atomics). */
edkm_status edkm_backward_dense(edkm_plan* plan, const uint16_t* w_bits,
                                const float* grad_w_tilde, float* grad_w, float* grad_c,
                                hipStream_t stream);

/* Timing hook (diagnostics).  The N-sized passes, one kernel launch each per
 * call (per launch group in the batched forms): */
enum {
    EDKM_PASS_HIST = 0,         /* init_unique: pattern histogram, reads 2 B/weight */
    EDKM_PASS_GATHER_WT = 1,    /* forward: W~ gather, 2 B + 4 B (16-bit out: 2 B) */
    EDKM_PASS_KEYED_GRAD = 2,   /* backward: keyed sum of dL/dW~, 2 B + 4 B */
    EDKM_PASS_GATHER_GRAD = 3,  /* backward: dL/dw gather, 2 B + 4 B + 4 B */
    /* Dense comparison path: one map evaluation over all N weights, k
     * exponentials per weight.  A call launches several; the events bracket
     * the last one of the call. */
    EDKM_PASS_DENSE_ITER = 4,   /* forward_dense: one centroid iteration, reads 2 B */
    EDKM_PASS_DENSE_BITER = 5,  /* backward_dense: one unrolled iteration, 2 B + 4 B + 4 B */
    EDKM_PASS_PALETTIZE = 6,    /* palettize: packed indices, 2 B + b/8 B */
    EDKM_PASS_INVERSE = 7       /* unique_inverse: inverse index, 2 B + 2 B */
};
/* When set (non-NULL), later calls on this plan record `start` on the stream
 * right before that pass's launch and `stop` right after it; in a batched call
 * the events of the first plan of each launch group are used.  The caller owns
 * the events (created with timing enabled) and reads them with
 * hipEventElapsedTime.  NULL events switch the hook off.  Host only. */
edkm_status edkm_plan_set_pass_events(edkm_plan* plan, int pass, hipEvent_t start, hipEvent_t stop);

/* Palettization: the compressed artefact of weight clustering, a lookup
 * table of k entries plus a b-bit index per weight (Sec. 2).  Each weight
 * takes the index of its nearest table entry,
 *   index_i = the j minimising |w_i - lut[j]|   (lowest j on ties),
 * decided in fp32 (w_i is exact in fp32; one fp32 subtraction per entry);
 * non-finite weights get index 0.  The indices are packed little-endian, b =
 * bits of the plan: index i occupies bits [b i, b i + b) of the output bit
 * stream, byte m holding stream bits 8m..8m+7 (least significant first);
 * bits past n b are zero.
 *   w_bits       device, n patterns (the plan's weight format)
 *   lut          device float[k]: the table, e.g. c_out of edkm_forward
 *   indices_out  device uint8[ceil(n b / 8)]
 * Needs no init_unique and leaves the plan's forward/backward state alone
 * (it uses its own part of the workspace).  Cost: one read of the keys and
 * one write of n b / 8 bytes. */
edkm_status edkm_palettize(edkm_plan* plan, const uint16_t* w_bits, const float* lut,
                           uint8_t* indices_out, hipStream_t stream);
/* Batched form: `count` matrices, each with its own plan, keys, table and
 * output, cut into launch groups of up to EDKM_LAUNCH_GROUP consecutive matrices with the same
 * bit width and weight format; each group is one table launch and one packing
 * launch.  Host arrays of `count` entries, none NULL.  Equivalent to calling
 * edkm_palettize on each. */
edkm_status edkm_palettize_batch(int count, edkm_plan* const* plans, const uint16_t* const* w_bits,
                                 const float* const* lut, uint8_t* const* indices_out,
                                 hipStream_t stream);

/* Palettization for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * edkm_palettize for one matrix of n weights (1..EDKM_MAX_N), bits in 1..4
 * and key_format EDKM_KEYS_FP16 or EDKM_KEYS_BF16, with the same inputs,
 * output and result, but no plan and no workspace.  Its per-pattern index
 * table lives in a device array of EDKM_NOALLOC_SCRATCH_BYTES that the
 * library holds on each GPU it runs on until the process ends; the call
 * allocates nothing (no hipMalloc, no allocating library routine).  The first
 * call on a device looks up that array's address there (hipGetSymbolAddress;
 * make one call on each device before capturing a graph if the capture mode
 * forbids that query).  Every call on one GPU uses the same array and
 * rewrites all of it, so nothing carries over between calls, but calls that
 * overlap on one GPU (other streams, other threads) race on it: serialise
 * them.  Errors: EDKM_ERR_ARG for a null pointer, n = 0 or above EDKM_MAX_N,
 * bits outside 1..4 or an unknown format (checked before any HIP call);
 * EDKM_ERR_HIP if the address lookup or a launch fails. */
#define EDKM_NOALLOC_SCRATCH_BYTES 65536
edkm_status edkm_palettize_noalloc(const uint16_t* w_bits, uint64_t n, int bits, int key_format,
                                   const float* lut, uint8_t* indices_out, hipStream_t stream);

/* The uniquification's two lists (Sec. 2.2): the distinct weight patterns
 * and, per weight, the index of its pattern among them, in ascending order of
 * the 16-bit key (the order of numpy.unique on the uint16 view, with
 * return_inverse).  Every pattern counts, Inf/NaN ones included, and +0 / -0
 * are distinct.  The forward and backward never need these lists (the key is
 * the table offset); this is for callers that store or ship the index list.
 *   w_bits       device, n patterns; must be the buffer given to init_unique
 *                (the distinct patterns come from its counts)
 *   unique_out   nullable, device uint16[65536]: entries 0 .. U-1 receive the
 *                U distinct patterns, ascending (U = num_unique of
 *                init_unique); later entries are left alone
 *   inverse_out  nullable, device uint16[n]: inverse_out[i] = the index of
 *                w_bits[i] in unique_out, so unique_out[inverse_out[i]] =
 *                w_bits[i]
 * At least one output must be given (EDKM_ERR_ARG otherwise).  Needs
 * init_unique on this plan and key buffer (EDKM_ERR_STATE otherwise); may be
 * called after forward or backward and leaves their state alone (it uses its
 * own part of the workspace).  Exact (integer).  Cost: one pass over the
 * 65,536 counts, and with inverse_out one read of the keys and one write of
 * 2 bytes per weight. */
edkm_status edkm_unique_inverse(edkm_plan* plan, const uint16_t* w_bits, uint16_t* unique_out,
                                uint16_t* inverse_out, hipStream_t stream);
/* Batched form: host arrays of `count` entries (the arrays and their entries
 * may be NULL where an output is not wanted, but each matrix needs one
 * output), cut into launch groups of up to EDKM_LAUNCH_GROUP consecutive
 * matrices; each group is one ranking launch and, if any matrix of the group
 * wants the inverse index, one N-sized launch.  Equivalent to calling
 * edkm_unique_inverse on each. */
edkm_status edkm_unique_inverse_batch(int count, edkm_plan* const* plans,
                                      const uint16_t* const* w_bits, uint16_t* const* unique_out,
                                      uint16_t* const* inverse_out, hipStream_t stream);

/* Keyed-gradient accumulators (the backward's keyed reduction).  AUTO, the
 * default, chooses per matrix at init_unique from how concentrated the
 * weight patterns are: 32-bit fixed point with returning LDS atomics when few
 * lanes of an atomic share a pattern (fp16 weights), 64-bit fixed point with
 * plain atomics when many do (bf16 weights, low-entropy data).  Both are exact
 * in the sense that no sum is lost; they differ in speed and in the last bits.
 * Limit of the 32-bit mode: its overflow carries are added to fp32 sums, which
 * stay exact while a pattern's same-sign gradient sum is below about 2^28
 * times a typical |gradient|.  AUTO picks the 32-bit mode only when every
 * pattern holds under 1.7% of the weights (at most 7.4e7 of 2^32), so it
 * never reaches that; forcing EDKM_KEYED_I32 on data where one pattern holds
 * more than 2^28 weights can lose precision.
 * The setting takes effect at the next init_unique on this plan.  Host only. */
enum {
    EDKM_KEYED_AUTO = -1,
    EDKM_KEYED_I32 = 0,
    EDKM_KEYED_U64 = 1
};
edkm_status edkm_plan_set_keyed_mode(edkm_plan* plan, int mode);

/* Diagnostics for the last EDKM_ERR_HIP returned on this plan: the HIP error
 * code (0 if none), the launch or runtime call that failed, and the HIP
 * runtime's description.  The strings are static.  Any output may be NULL. */
edkm_status edkm_plan_hip_error(const edkm_plan* plan, int* code, const char** step,
                                const char** message);

/* Static string for a status code. */
const char* edkm_status_str(edkm_status status);

#ifdef __cplusplus
}
#endif
#endif /* EDKM_H */
