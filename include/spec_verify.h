/*
 * spec_verify.h -- C ABI of the fused speculative-sampling verification step
 * for AMD Instinct MI355X (gfx950).
 *
 * The operation is the verification part of speculative sampling as treated
 * in "Optimized Speculative Sampling for GPU Hardware Accelerators"
 * (arXiv 2406.11016):
 *
 *   - Sec. 3.1, eq. (1): drafted token x_c (c = 0..gamma-1) is accepted iff
 *     r_c <= tau_c = min(1, p_c(x_c) / q_c(x_c)); the scan stops at the first
 *     rejection;
 *   - Sec. 3.1, eqs. (2)-(3): after a rejection at position L the next token
 *     is drawn from max(0, p_L - q_L) / sum_x max(0, p_L - q_L);
 *   - Sec. 3.2.2, eq. (4): in the exact mode p and q are the softmax of the
 *     target and draft logits;
 *   - Sec. 3.2.2, eq. (5): in the sigmoid mode they are replaced by
 *     sigma((z - alpha) / (beta - alpha)), element-wise and unnormalised, with
 *     the same acceptance test and residual.
 *
 * Points the paper leaves open are fixed as follows:
 *   - when all gamma drafts are accepted the next token is drawn from the
 *     target row gamma (exact: softmax; sigmoid: p_hat_gamma / sum p_hat_gamma);
 *   - draws use caller-supplied uniforms: uniforms[b, c] is r_c for c < gamma
 *     and uniforms[b, gamma] drives the final draw, which is the first index j
 *     with cumsum(a)[j] > u * sum(a) (inverse CDF over token ids in order);
 *   - a tie r_c == tau_c accepts; q_c(x_c) == 0 gives tau_c = 1;
 *   - if the residual mass is zero after a rejection (possible only in the
 *     sigmoid mode) the next token is drawn from row L of the target instead;
 *   - the temperature T divides the logits before either mode;
 *   - token ids are 0-based.
 *
 * Layout.  All tensors are dense, row-major, and live in device memory:
 *   draft_logits   [B, gamma,   V]  dtype
 *   target_logits  [B, gamma+1, V]  dtype
 *   draft_tokens   [B, gamma]       int32, the drafted tokens x_c
 *   uniforms       [B, gamma+1]     fp32 in [0, 1)
 *   accepted_len   [B]              int32 out, L in [0, gamma]
 *   next_token     [B]              int32 out, in [0, V)
 * Rows need no particular alignment; rows starting at a 4-byte aligned
 * address (every fp32 row, 16-bit rows of even V) are read with 128-bit loads.
 *
 * Ownership and concurrency.  Every pointer is owned by the caller.  The
 * library never allocates device memory and never prints; only
 * spec_verify_workspace_check and the decoding loop's step wait for the
 * stream.  Inputs are only read; outputs and the workspace are overwritten.  A call enqueues its
 * kernels on `stream` and returns without waiting: SV_OK means "launched".
 * The workspace must be zero-filled once before its first use (for example
 * with spec_verify_workspace_init); every call leaves it zero-filled again.
 * It carries the hand-off between the workgroups of the single launch a call
 * makes.  Calls that share a workspace must be ordered (same stream, or
 * synchronised); concurrent calls need separate workspaces.  There is no
 * mutable global state other than spec_verify_exact_static's per-device
 * workspace lookup (guarded by a mutex): the functions are reentrant and
 * thread-safe.
 *
 * Errors.  Invalid arguments are detected on the host before anything is
 * launched and return a negative status.  Bad data found on the device --
 * a drafted token outside [0, V), a read row whose distribution is not
 * finite (a NaN logit; in the exact mode also a +inf logit or a row that is
 * entirely -inf), or a non-finite or zero final mass -- writes the sentinel
 * accepted_len[b] = next_token[b] = -1 for that batch element only.  In the
 * exact mode the rows read are the target and draft rows 0..L and, when
 * L == gamma, target row gamma; in the sigmoid mode they are the logits at
 * the drafted tokens of rows 0..L and the full row(s) the next token is drawn
 * from.  Logits must satisfy |z| / T < 2.3e38 (so that z * log2(e) / T is
 * finite).
 *
 * Timed-out waits.  The workgroups of a launch hand results to each other
 * through the workspace, and every such wait is bounded (about 0.1 s) so that
 * every wave exits even if a producer never runs.  A wait that gives up sets
 * the workspace's sticky error flag (spec_verify_workspace_check reads it),
 * and the outputs of that call are not valid: every output is still written,
 * with -1 or a value in its range, but an element's two outputs may come
 * from different workgroups.  Results that arrive after their reader gave up
 * stay in the workspace, so every later call on a workspace whose flag is set
 * writes the sentinel -1 to every output, until the workspace is zero-filled
 * again (spec_verify_workspace_init).  No wait times out in normal
 * operation.
 */
#ifndef SPEC_VERIFY_H
#define SPEC_VERIFY_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Storage type of the logits.  (In C++ the enum has the fixed underlying
 * type int32_t, so that any value a C caller passes is a valid value of the
 * type and is rejected by the checks instead of being undefined.) */
typedef enum sv_dtype
#ifdef __cplusplus
    : int32_t
#endif
{
    SV_F32 = 0,   /* IEEE binary32 */
    SV_F16 = 1,   /* IEEE binary16 */
    SV_BF16 = 2   /* bfloat16 (upper half of a binary32) */
} sv_dtype_t;

typedef enum sv_status {
    SV_OK = 0,
    SV_ERR_NULL = -1,       /* a required pointer is NULL */
    SV_ERR_SHAPE = -2,      /* B < 1, gamma < 1 or > SV_MAX_GAMMA, V < 1, or sizes overflow */
    SV_ERR_DTYPE = -3,      /* unknown sv_dtype_t */
    SV_ERR_PARAM = -4,      /* temperature not finite and > 0; alpha/beta not finite with alpha < beta */
    SV_ERR_WORKSPACE = -5,  /* workspace smaller than spec_verify_workspace_bytes() or not 16-byte aligned */
    SV_ERR_HIP = -6,        /* a HIP launch failed (hipGetLastError after the launches), or a HIP
                               call of the decoding loop or of spec_verify_workspace_check failed */
    SV_ERR_ALLOC = -7,      /* the decoding loop could not allocate its host object */
    SV_ERR_TIMEOUT = -8     /* the workspace's error flag is set: a wait between workgroups timed out
                               (in this call or an earlier one since the workspace was zero-filled);
                               outputs are not valid until the workspace is re-initialised */
} sv_status_t;

/* Largest number of drafted tokens per step supported by one call. */
#define SV_MAX_GAMMA 128

/*
 * Bytes of device workspace a call with these sizes needs (the same value
 * serves both modes).  Returns 0 for invalid sizes, including vocabularies
 * above 2^20 (fp32) or 2^21 (fp16 / bf16) entries.  The workspace holds the
 * per-chunk normaliser partials (exact mode), one copy of each batch
 * element's decision per workgroup that reads it, the per-chunk masses of
 * the final distribution and the early exit's per-position hand-off words,
 * after a 256-byte header.  Header words (32-bit, zero in a zero-filled
 * workspace): byte offset 4 is the sticky error flag, set when a wait between
 * workgroups times out (see "Timed-out waits" above); byte offset 8, when
 * nonzero, replaces the default bound on every wait by that many polls (a test
 * hook, to force the timeout path from the host).
 */
size_t spec_verify_workspace_bytes(int32_t batch, int32_t gamma, int32_t vocab, sv_dtype_t dtype);

/*
 * Zero-fills `workspace_bytes` bytes of `workspace` on `stream` with a fill
 * kernel (no memset node, so the call may be captured in a graph).
 */
sv_status_t spec_verify_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * WAITS for `stream` to finish (unlike every other call here), then reads the
 * workspace's sticky error flag: SV_OK if it is clear, SV_ERR_TIMEOUT if a wait
 * between workgroups timed out in a call on this workspace since it was last
 * zero-filled (the outputs of that call and of every later one are then not
 * valid), SV_ERR_HIP if a HIP call failed.  SV_ERR_NULL for a NULL workspace,
 * SV_ERR_WORKSPACE if it is smaller than its 256-byte header or not 16-byte
 * aligned.
 */
sv_status_t spec_verify_workspace_check(const void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Exact mode (Sec. 3.1 with the softmax of eq. (4)): softmax of every target
 * and draft row at temperature T, the acceptance test of eq. (1) at the
 * drafted tokens, the first-rejection scan, and the inverse-CDF draw from the
 * residual of eqs. (2)-(3) (or from target row gamma when all drafts are
 * accepted).  The result equals the plain definition up to floating-point
 * rounding (fp32 element arithmetic, fp64 reductions).
 */
sv_status_t spec_verify_exact(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                              const int32_t* draft_tokens, const float* uniforms,
                              int32_t batch, int32_t gamma, int32_t vocab, float temperature,
                              int32_t* accepted_len, int32_t* next_token,
                              void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Exact mode with an early exit: the same result as spec_verify_exact,
 * computed so that the logit rows a batch element does not need are mostly
 * not read.  Its row chunks are twice as long as spec_verify_exact's, so its
 * row normalisers can differ from that call's in the last bits: a decision
 * can differ only where a uniform lies within that rounding of its
 * threshold.  Sec. 3.1 stops the acceptance scan at
 * the first rejection L, so the rows of positions after L (and target row
 * gamma when L < gamma) play no part in the result.  The rows stream in draft
 * order (stage c: target row c and draft row c of every batch element), each
 * position's test of eq. (1) is made once its two rows' normalisers are in
 * (one stage later), and the tiles of a stage about 56 MB of stream later (at
 * least two stages) skip their row when their element has already rejected a
 * draft.
 * Worth it when B is large and drafts are often rejected; when nearly every
 * draft is accepted it streams the same bytes as spec_verify_exact through
 * more hand-offs.  Batches whose stream is too short for any decision row to
 * be skipped (a stage of 2 B V s bytes: the two-stage minimum reaches no
 * decision row when gamma <= 2, and about 56 MB of stream reaches none when
 * 56e6 / (2 B V s) > gamma - 1), and launches past 2^31 workgroups, run
 * spec_verify_exact's single pass.
 * Arguments, layout, ownership, workspace and errors as spec_verify_exact.
 */
sv_status_t spec_verify_exact_early_exit(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                         const int32_t* draft_tokens, const float* uniforms,
                                         int32_t batch, int32_t gamma, int32_t vocab, float temperature,
                                         int32_t* accepted_len, int32_t* next_token,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Size of the static device workspace of spec_verify_exact_static, per GPU. */
#define SV_STATIC_WORKSPACE_BYTES (8u << 20)

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * spec_verify_exact with the library's own static workspace instead of a
 * caller's.  Same arguments, layout, results and errors as spec_verify_exact,
 * without workspace / workspace_bytes.
 *
 * The workspace is a SV_STATIC_WORKSPACE_BYTES (8 MiB) array in the library's
 * device code, one per GPU, held until the process ends; nothing is allocated
 * or freed.  The first call on a device (the current device, which must own
 * `stream`) looks it up and zero-fills it with a fill kernel on `stream`.
 * Every call on a GPU shares that GPU's array and leaves it zero-filled, so
 * calls that overlap in time on one GPU (other streams, other threads) race
 * and give wrong results: order them.  After a timed-out wait (see
 * "Timed-out waits") every later call writes the sentinel -1 to every output
 * until a call passes `reset` nonzero, which zero-fills the array on `stream`
 * before the step.  Sizes whose spec_verify_workspace_bytes() exceeds
 * SV_STATIC_WORKSPACE_BYTES (for example B > ~1400 at gamma = 8,
 * V = 128,256) return SV_ERR_WORKSPACE before anything is launched.
 */
sv_status_t spec_verify_exact_static(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                     const int32_t* draft_tokens, const float* uniforms,
                                     int32_t batch, int32_t gamma, int32_t vocab, float temperature,
                                     int32_t* accepted_len, int32_t* next_token, int32_t reset,
                                     hipStream_t stream);

/*
 * Sigmoid mode (Sec. 3.2.2, eq. (5)): p_hat = sigma((z_p / T - alpha) / (beta - alpha))
 * and q_hat likewise replace the softmax; tau_hat = min(1, p_hat / q_hat) at
 * the drafted tokens; after a rejection at L the next token is drawn from
 * max(0, p_hat_L - q_hat_L) normalised.  Only the logits at the drafted
 * tokens and the row(s) the next token is drawn from are read.  The paper
 * uses alpha = -beta = -1e3 (speech) and -1e4 (summarisation).
 */
sv_status_t spec_verify_sigmoid(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                const int32_t* draft_tokens, const float* uniforms,
                                int32_t batch, int32_t gamma, int32_t vocab, float temperature,
                                float alpha, float beta,
                                int32_t* accepted_len, int32_t* next_token,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Probe variants for testing: the same computation as spec_verify_exact /
 * spec_verify_sigmoid, additionally writing any of these that is non-NULL
 * (device pointers):
 *   tau_out      [B, gamma]      fp64: tau_c of eq. (1) (or its sigmoid form)
 *                                for every c (NaN where a row is unreadable);
 *   weight_out   [B, V]          fp32: the unnormalised weights a(x) of the
 *                                distribution the next token is drawn from;
 *   mass_out     [B]             fp64: their sum b;
 *   lognorm_out  [B, 2*gamma+1]  fp64 (exact mode only): log sum_x exp(z_r(x)/T)
 *                                of target rows 0..gamma, then draft rows
 *                                0..gamma-1.
 * Rows with the sentinel leave weight_out and mass_out unspecified.
 */
sv_status_t spec_verify_exact_probe(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                    const int32_t* draft_tokens, const float* uniforms,
                                    int32_t batch, int32_t gamma, int32_t vocab, float temperature,
                                    int32_t* accepted_len, int32_t* next_token,
                                    void* workspace, size_t workspace_bytes, hipStream_t stream,
                                    double* tau_out, float* weight_out, double* mass_out,
                                    double* lognorm_out);

sv_status_t spec_verify_sigmoid_probe(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                      const int32_t* draft_tokens, const float* uniforms,
                                      int32_t batch, int32_t gamma, int32_t vocab, float temperature,
                                      float alpha, float beta,
                                      int32_t* accepted_len, int32_t* next_token,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream,
                                      double* tau_out, float* weight_out, double* mass_out);

/*
 * Ragged variants: batch element b drafted gammas[b] tokens (1 <= gammas[b]
 * <= gamma_max; `gammas` is a device array of B int32).  The tensors keep the
 * padded shapes of gamma_max -- draft [B, gamma_max, V], target
 * [B, gamma_max + 1, V], draft_tokens [B, gamma_max], uniforms
 * [B, gamma_max + 1] -- and element b uses its draft rows 0..gammas[b]-1,
 * target rows 0..gammas[b], tokens and acceptance uniforms 0..gammas[b]-1,
 * and uniforms[b, gammas[b]] for the final draw; everything beyond is never
 * read.  Each element is exactly the step of spec_verify_exact /
 * spec_verify_sigmoid at its own gamma (Sec. 3.1 treats each sequence's drafts
 * independently); accepted_len[b] lies in [0, gammas[b]].  An element whose
 * gammas[b] lies outside 1 .. gamma_max gets the sentinel -1 in both outputs.
 * The workspace is that of spec_verify_workspace_bytes(batch, gamma_max, ...).
 * `gammas` NULL returns SV_ERR_NULL.
 */
sv_status_t spec_verify_exact_ragged(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                     const int32_t* draft_tokens, const float* uniforms, const int32_t* gammas,
                                     int32_t batch, int32_t gamma_max, int32_t vocab, float temperature,
                                     int32_t* accepted_len, int32_t* next_token,
                                     void* workspace, size_t workspace_bytes, hipStream_t stream);

sv_status_t spec_verify_sigmoid_ragged(const void* draft_logits, const void* target_logits, sv_dtype_t dtype,
                                       const int32_t* draft_tokens, const float* uniforms, const int32_t* gammas,
                                       int32_t batch, int32_t gamma_max, int32_t vocab, float temperature,
                                       float alpha, float beta,
                                       int32_t* accepted_len, int32_t* next_token,
                                       void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Decoding loop (Sec. 4, hyperparameters: the number of drafts starts at 5,
 * grows by 2 after an iteration in which every draft was accepted and
 * otherwise shrinks by 1; here it stays within 1 .. gamma_max, and with
 * several batch elements every element must accept every draft to grow).
 *
 * The caller owns static buffers sized for gamma_max and, before each
 * iteration, writes the iteration's inputs into their leading parts as the
 * dense tensors of spec_verify_exact / spec_verify_sigmoid at that gamma
 * (draft [B, gamma, V] at `draft`, target [B, gamma+1, V] at `target`,
 * tokens [B, gamma], uniforms [B, gamma+1]), on `stream` or ordered before
 * it.  spec_verify_loop_step then runs the step, copies accepted_len and
 * next_token into `host_out` (pinned host memory, [2B] int32: the accepted
 * lengths, then the next tokens), WAITS for the stream to finish (the host
 * needs L to choose the next gamma and the tokens to append), and writes the
 * next gamma.  With use_graphs the step and the three copies are captured
 * into a HIP graph the first time each gamma is used and replayed afterwards
 * (on ROCm 7 replaying this one-kernel graph measured slower than launching
 * it directly, so direct launch is the better default).
 *
 * After the wait the step also reads the workspace's sticky error flag (copied
 * to pinned memory with the outputs) and returns SV_ERR_TIMEOUT, leaving
 * *next_gamma unwritten, if it is set.
 *
 * Early exit (exact mode; Sec. 3.1 stops at the first rejection):
 * `early_exit` 0 runs every step through spec_verify_exact, 1 through
 * spec_verify_exact_early_exit, 2 chooses per step from the previous step's
 * acceptance: the early exit when the mean accepted length over the batch
 * (sentinels counting 0) was below half of that step's gamma, the single pass
 * otherwise and at the first step.  Both give the same outputs; the early
 * exit is faster when most elements reject early and slower when they
 * accept most drafts.  spec_verify_loop_last_early_exit reports the choice
 * of the last step (1: early exit, 0: single pass, -1: no step yet).
 *
 * Ownership: every pointer in the descriptor is the caller's and must stay
 * valid until spec_verify_loop_destroy; the loop allocates only its host
 * object, one pinned 4-byte word for the flag (at the first step) and the
 * graphs.  The workspace must hold
 * spec_verify_workspace_bytes(batch, g, vocab, dtype) for every g up to
 * gamma_max (zero-filled before the first iteration; each iteration leaves it
 * zero-filled).  One loop must not be stepped from two threads at once.
 * Errors: SV_ERR_NULL, SV_ERR_SHAPE, SV_ERR_PARAM (mode not 0/1, early_exit
 * not 0-2, gamma out of 1 .. gamma_max), SV_ERR_WORKSPACE, SV_ERR_ALLOC at creation; the
 * verification's own errors, SV_ERR_HIP and SV_ERR_TIMEOUT at a step.
 */
typedef struct sv_loop sv_loop;

typedef struct sv_loop_desc {
    int32_t mode;                 /* 0: exact (spec_verify_exact), 1: sigmoid (spec_verify_sigmoid) */
    sv_dtype_t dtype;
    int32_t batch, gamma_max, vocab;
    float temperature, alpha, beta;   /* alpha, beta: sigmoid mode only */
    void* draft;                  /* device, B * gamma_max * V logits */
    void* target;                 /* device, B * (gamma_max + 1) * V logits */
    int32_t* tokens;              /* device, B * gamma_max */
    float* uniforms;              /* device, B * (gamma_max + 1) */
    int32_t* accepted_len;        /* device [B] */
    int32_t* next_token;          /* device [B] */
    int32_t* host_out;            /* pinned host [2B] */
    void* workspace;
    size_t workspace_bytes;
    hipStream_t stream;
    int32_t use_graphs;           /* nonzero: one captured graph per gamma (and entry point) */
    int32_t early_exit;           /* exact mode: 0 never, 1 always, 2 from the previous step's acceptance */
} sv_loop_desc_t;

sv_status_t spec_verify_loop_create(const sv_loop_desc_t* desc, sv_loop** loop);
sv_status_t spec_verify_loop_step(sv_loop* loop, int32_t gamma, int32_t* next_gamma);
sv_status_t spec_verify_loop_destroy(sv_loop* loop);
int32_t spec_verify_loop_last_early_exit(const sv_loop* loop);

/* Static description of a status code. */
const char* spec_verify_status_string(sv_status_t status);

#ifdef __cplusplus
}
#endif

#endif /* SPEC_VERIFY_H */
