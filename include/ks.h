/*
 * ks.h -- C ABI of the MI355X (gfx950) Kronecker-sparse matrix multiplication
 * library (libks.so).
 *
 * Operation (paper, Section 1 "Scope of this work"; Definition 2.1):
 *   K is a KS matrix of pattern (a, b, c, d): an (a*b*d) x (a*c*d) matrix whose
 *   support lies in I_a (x) 1_{b x c} (x) I_d.  For a batch X of `batch` row
 *   vectors of length N = a*c*d the library computes Y = X K^T, whose rows have
 *   length M = a*b*d.  Every (i, j) in [a] x [d] owns the output rows
 *   i*b*d + k*d + j (k < b) and the input columns i*c*d + l*d + j (l < c)
 *   (Section 4.1, Algorithm 2); these sets partition [M] and [N], so every
 *   element of Y is written exactly once and Y need not be initialised.
 *
 * Packed values (Appendix A.1 "(ad, b, c)" storage; Section 4.2 assumes K is
 * pre-arranged offline):  K_values holds a*d dense b x c blocks, row-major,
 *     K_values[((i*d + j)*b + k)*c + l] = K[i*b*d + k*d + j, i*c*d + l*d + j].
 *
 * Layouts (Section 2.2), all row-major and densely packed, no leading
 * dimensions:
 *   KS_LAYOUT_BSF  batch-size-first: X is (batch, N), Y is (batch, M);
 *   KS_LAYOUT_BSL  batch-size-last:  X is (N, batch), Y is (M, batch).
 *
 * Types: X, K_values and Y share one storage type (fp32, bf16 or fp16), or,
 * for KS_FP8_E4M3, X and K_values are FP8 E4M3 and Y is bf16; products are
 * accumulated in fp32 and the result is rounded to Y's type with
 * round-to-nearest-even (the paper's conclusion names lower precision as its
 * kernel's open limitation).
 *
 * Ownership: every pointer argument except `pattern` arrays and factor lists is
 * a device pointer owned by the caller; the library allocates no device memory.
 * The only library-owned state is a host-side plan cache (thread-safe).
 *
 * Execution: work is enqueued asynchronously on `stream` (a hipStream_t; NULL
 * is the legacy default stream) with the usual stream-ordering rules.  All
 * argument checks happen on the host before anything is enqueued; on any error
 * nothing is enqueued and the contents of Y are unspecified.  A failure reported
 * by the HIP runtime at launch returns KS_ERR_HIP and its hipError_t can be read
 * with ks_last_hip_error() on the same thread.
 */
#ifndef KS_H_
#define KS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    KS_LAYOUT_BSF = 0, /* batch-size-first: X (batch, N), Y (batch, M) */
    KS_LAYOUT_BSL = 1  /* batch-size-last:  X (N, batch), Y (M, batch) */
} ks_layout_t;

typedef enum {
    KS_F32 = 0,     /* IEEE binary32 */
    KS_BF16 = 1,    /* bfloat16 */
    KS_F16 = 2,     /* IEEE binary16 */
    KS_FP8_E4M3 = 3 /* X and K_values in OCP FP8 E4M3 ("E4M3FN": bias 7, no
                       infinities, max 448); Y (and a bias) in bfloat16.
                       Single factors only (ks_chain: KS_ERR_UNSUPPORTED). */
} ks_dtype_t;

typedef enum {
    KS_OK = 0,
    KS_ERR_INVALID_PATTERN = 1, /* a, b, c or d < 1, or a size overflows int64 */
    KS_ERR_INVALID_ARG = 2,     /* NULL pointer, batch < 0, bad factor count */
    KS_ERR_DIM_MISMATCH = 3,    /* chain: a_f*c_f*d_f != a_{f+1}*b_{f+1}*d_{f+1} */
    KS_ERR_ALIAS = 4,           /* X and Y (or a workspace) overlap */
    KS_ERR_UNSUPPORTED = 5,     /* unknown dtype or layout, or a size beyond the supported range */
    KS_ERR_WORKSPACE = 6,       /* chain workspace missing or too small */
    KS_ERR_HIP = 7,             /* the HIP runtime reported an error at launch */
    KS_ERR_SCRATCH_LIMIT = 8    /* ks_chain_noalloc: intermediates exceed its fixed scratch array */
} ks_status_t;

/* Output activation of ks_matmul_bias_act. */
typedef enum {
    KS_ACT_NONE = 0,
    KS_ACT_GELU = 1 /* exact GELU: x * Phi(x) = 0.5 x (1 + erf(x / sqrt 2)) */
} ks_act_t;

/* One factor of a chain: its pattern and its packed values (device pointer,
 * layout as K_values above). */
typedef struct {
    int64_t a, b, c, d;
    const void *K_values;
} ks_factor_t;

/*
 * Y = X K^T for one KS factor of pattern (a, b, c, d)  (Section 1; Algorithm 2
 * of Section 4.1 is the tiling the kernels follow).
 *   K_values  device, a*d*b*c elements, packed as described above.
 *   X         device, batch*a*c*d elements in `layout`.
 *   Y         device, batch*a*b*d elements in `layout`; fully overwritten.
 *             Must not overlap X (KS_ERR_ALIAS).
 *   batch     number of vectors; 0 enqueues nothing and returns KS_OK.
 * Any element-aligned pointer is accepted; the planner picks narrower memory
 * accesses when a pointer or a row is not 16-byte aligned.  Sizes: every tensor
 * must have fewer than 2^31 elements (KS_ERR_UNSUPPORTED otherwise).
 */
ks_status_t ks_matmul(int64_t a, int64_t b, int64_t c, int64_t d,
                      const void *K_values, const void *X, void *Y,
                      int64_t batch, int layout, int dtype, void *stream);

/*
 * Y = act(X K^T + bias): ks_matmul with the bias and activation of a
 * Transformer MLP layer applied in the kernels' epilogue, in fp32 before the
 * rounding to the storage type (paper appendix, ViT-S/16 submodule table:
 * "Linear + bias" rows and the feed-forward block Linear + GELU).
 *   bias  device, a*b*d elements of `dtype`, one per output feature m (the
 *         column of Y in BSF, its row in BSL), added to every batch entry;
 *         NULL for no bias.  Must not overlap Y (KS_ERR_ALIAS).
 *   act   KS_ACT_NONE or KS_ACT_GELU (other values: KS_ERR_UNSUPPORTED).
 * Every other argument, the result layout and the errors are ks_matmul's;
 * ks_matmul(...) is ks_matmul_bias_act(..., NULL, KS_ACT_NONE, ...).
 */
ks_status_t ks_matmul_bias_act(int64_t a, int64_t b, int64_t c, int64_t d,
                               const void *K_values, const void *bias, int act,
                               const void *X, void *Y, int64_t batch,
                               int layout, int dtype, void *stream);

/*
 * Bytes of device workspace ks_chain needs for these factors: 0 for a single
 * factor and for chains that run fused in both layouts (see ks_chain), else
 * one (two factors) or two (more) intermediate buffers.  Returns 0 as well for invalid
 * arguments; ks_chain reports those.  The answer depends on this thread's
 * ks_force_variant / ks_force_chain_fusion settings, as ks_chain's plan does.
 */
size_t ks_chain_workspace_bytes(const ks_factor_t *factors, int nfactors,
                                int64_t batch, int dtype);

/*
 * Y = X (K_1 K_2 ... K_L)^T for the L = nfactors factors listed in product
 * order (Section 1, Figure 1; Appendix B.1, Table 5): K_L is applied first,
 * then K_{L-1}, ..., K_1.  Neighbouring factors must satisfy
 *     a_f * c_f * d_f == a_{f+1} * b_{f+1} * d_{f+1}   (KS_ERR_DIM_MISMATCH).
 * X has batch*a_L*c_L*d_L elements and Y batch*a_1*b_1*d_1, both in `layout`.
 * Chains of two to 24 factors whose blocks are all at most 8 x 8 -- e.g. the
 * butterfly factors of a transform of size up to 1024 -- or all square b x b
 * with one b in {16, 32, 48, 64} -- e.g. Monarch factors; batch-size-first,
 * and batch-size-last in fp32 with b <= 32 and width <= 1024 -- and whose
 * widest vector (times 16 or 32 batch columns of fp32, plus the small-block
 * form's factor-value buffer) fits in 160 KB of LDS, run as one fused kernel:
 * each workgroup keeps 16 or 32 batch columns of the intermediate vectors in
 * LDS in fp32 from the first factor to the last, so X is read once, Y is
 * written once and no workspace is used.  Other chains run
 * factor by factor
 * (one ks_matmul each); their intermediates are stored in `dtype` in the
 * caller's `workspace` (device, at least ks_chain_workspace_bytes(...) bytes,
 * not overlapping X or Y).  ks_chain_describe tells which applies.
 * Factor f's K_values are device pointers; the factor array itself is host
 * memory and may be freed when the call returns.
 */
ks_status_t ks_chain(const ks_factor_t *factors, int nfactors,
                     const void *X, void *Y, int64_t batch, int layout, int dtype,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * Fixed device scratch of ks_chain_noalloc, in bytes per GPU (64 MiB: the
 * intermediates of a 10-factor chain of width 1024 at batch 8192 in fp32, or
 * of a 2-factor chain of width 1024 at batch 16384 in fp32).
 */
#define KS_CHAIN_NOALLOC_MAX_WORKSPACE ((size_t)64 << 20)

/*
 * ks_chain without a workspace argument, for callers that cannot allocate
 * device memory (code under stream capture, serving loops, harnesses that
 * forbid allocation): the intermediates go to a fixed array of
 * KS_CHAIN_NOALLOC_MAX_WORKSPACE bytes inside the library (one copy per GPU,
 * allocated when the library's code object is loaded on that GPU and held
 * until the process ends).  The call itself allocates nothing.
 *   Arguments, results and errors are those of ks_chain, plus
 *   KS_ERR_SCRATCH_LIMIT when ks_chain_workspace_bytes(...) for these
 *   arguments exceeds the fixed size (nothing is enqueued then).
 *   The array's device address is looked up on the first call on each GPU
 *   (the current device); a failure there returns KS_ERR_HIP.
 * All calls on one GPU share its array: calls that may run at the same time on
 * one GPU (different streams or threads without ordering) race on it; calls
 * ordered on one stream do not.  Nothing in the array needs to start at zero.
 */
ks_status_t ks_chain_noalloc(const ks_factor_t *factors, int nfactors,
                             const void *X, void *Y, int64_t batch, int layout,
                             int dtype, void *stream);

/* The fixed scratch size of ks_chain_noalloc in bytes
 * (KS_CHAIN_NOALLOC_MAX_WORKSPACE). */
size_t ks_chain_noalloc_max_workspace(void);

/*
 * How ks_chain would run these arguments: writes "fused ..." (one kernel:
 * "fused" radix passes of small blocks, "fused-bfly" the dyadic butterfly in
 * two register passes, "fused-mfma" square blocks on the MFMAs; LDS bytes,
 * grid) or "unfused ... workspace=<bytes>" into `buf` (host, `len`
 * bytes, NUL-terminated).  Pure host call.  Returns KS_OK or the status
 * ks_chain would return for invalid factors, dtype or layout.
 */
ks_status_t ks_chain_describe(const ks_factor_t *factors, int nfactors,
                              int64_t batch, int layout, int dtype,
                              char *buf, size_t len);

/*
 * mode 0: chains on this thread always run factor by factor (one ks_matmul
 * per factor, with the caller's workspace); any other value restores the
 * automatic choice.  For testing and measuring both paths on the same inputs.
 */
void ks_force_chain_fusion(int mode);

/*
 * Host-side check of the fused kernel ks_chain would run for these arguments
 * (16-byte-aligned stand-in buffers): replays every workgroup's tile loads
 * and stores and every factor's work units on the CPU and checks that all
 * global accesses stay inside X and Y, every LDS row is inside its buffer,
 * each factor writes each element of its output exactly once (in place only
 * where a unit reads exactly the rows it writes), and every element of Y is
 * stored once.  Writes "ok", "not fused" or the first violation into
 * `report` (host, `len` bytes).  Enqueues nothing.  Returns KS_OK,
 * KS_ERR_UNSUPPORTED on a violation, or the status ks_chain_describe returns.
 */
ks_status_t ks_chain_verify(const ks_factor_t *factors, int nfactors,
                            int64_t batch, int layout, int dtype,
                            char *report, size_t len);

/* Human-readable name of a status code (static string). */
const char *ks_status_string(int status);

/* hipError_t behind the last KS_ERR_HIP returned on the calling thread
 * (0 if none). */
int ks_last_hip_error(void);

/*
 * Describe the plan (kernel variant and launch shape) the library would use for
 * ks_matmul with these arguments.  Writes a NUL-terminated string of at most
 * `len` bytes into `buf` (host memory).  Pure host call: enqueues nothing.
 * Returns KS_OK, or the status ks_matmul would return for these arguments.
 */
ks_status_t ks_plan_describe(int64_t a, int64_t b, int64_t c, int64_t d,
                             int64_t batch, int layout, int dtype,
                             char *buf, size_t len);

/*
 * Force the kernel variant used by later ks_matmul calls on this thread:
 * variant < 0 restores automatic planning; otherwise the numbering of
 * ks_plan_describe's "variant=" field.  A forced variant that cannot run the
 * given arguments makes ks_matmul return KS_ERR_UNSUPPORTED.  Used for tuning
 * and for testing every kernel on the same inputs.
 */
void ks_force_variant(int variant);

/*
 * Host-side check of the plan ks_matmul would use for these arguments (with
 * 16-byte-aligned buffers and the variant forced on this thread, if any):
 * replays every thread's address arithmetic on the CPU and checks that all
 * reads and writes stay in bounds and that every element of Y is written
 * exactly once (the row sets of Section 4.1 partition the output).  Enqueues
 * nothing.  Cost is proportional to batch*M; meant for tests and tuning.
 * Writes "ok" or the first violation into `report` (host, `len` bytes).
 * Returns KS_OK, KS_ERR_UNSUPPORTED on a violation or missing plan, or the
 * status ks_matmul would return for these arguments.
 */
ks_status_t ks_plan_verify(int64_t a, int64_t b, int64_t c, int64_t d,
                           int64_t batch, int layout, int dtype,
                           char *report, size_t len);

#ifdef __cplusplus
}
#endif

#endif /* KS_H_ */
