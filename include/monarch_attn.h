/*
 * monarch_attn.h -- C ABI of the MonarchAttention forward pass on MI355X (gfx950).
 *
 * MonarchAttention (Yaras et al., "MonarchAttention: Zero-Shot Conversion to
 * Fast, Hardware-Aware Structured Attention") replaces softmax(Q K^T / sqrt(d))
 * by a Monarch matrix M = P^T B (Sec. 2, "Monarch Matrices"), whose
 * block-diagonal factors L and R are found by T alternating closed-form
 * maximisations of the variational softmax objective (Sec. 3, eqs. R_update,
 * L_update, beta_r, beta_l), and returns O = M V through the two-step Monarch
 * product (eq. monarch_multiply).  L and R are never written to memory: only
 * the states alpha_R, c_R, alpha_L, c_L of the Implementation paragraph of
 * Sec. 3 (and Y) cross between kernels.
 *
 * Index convention (0-based): with N = m * b, query row l*b + j is Qbar[j][l]
 * and key/value row k*b + i is Kbar[k][i] / Vbar[k][i]; R[k][j][:] is a
 * softmax over i and L[j][:][l] a softmax over k.  The scores are scaled by
 * 1/sqrt(d).  L starts at the identity and R is updated before L in each of
 * the T steps (Sec. 3; Appendix "Naive Algorithm").
 *
 * All functions are plain C, thread-safe, and never throw.
 */
#ifndef MONARCH_ATTN_H
#define MONARCH_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Element types of q, k, v and out.  bf16/fp16 run the matrix products on
 * MFMA with fp32 accumulation; all softmax statistics and the normalisers
 * c_R, c_L are fp32.  fp32 runs fp32 MFMA throughout.  With 16-bit types
 * the states are rounded to the element type at every step, and over many
 * steps the iteration amplifies that rounding as much as it amplifies one
 * rounding of its inputs (a few 1e-2 relative at T = 16-64 on random
 * inputs, near 5e-3 for T of 1 to 4).  16-bit calls therefore take at most
 * MONARCH_ATTN_MAX_T_16BIT steps in the forward pass and
 * MONARCH_ATTN_MAX_T_16BIT_BWD in the gradient, the counts up to which
 * their 2e-2 (forward) and 3e-2 (gradient) relative accuracy has been
 * validated; fp32 takes up to 64 (32 for the gradient). */
typedef enum { MA_F32 = 0, MA_BF16 = 1, MA_F16 = 2 } ma_dtype;

#define MONARCH_ATTN_MAX_T_16BIT 4
#define MONARCH_ATTN_MAX_T_16BIT_BWD 4

typedef enum {
    MA_OK = 0,
    MA_EINVAL = 1,        /* malformed arguments: nothing was launched            */
    MA_EUNSUPPORTED = 2,  /* well-formed but outside the supported shapes         */
    MA_EHIP = 3,          /* a HIP runtime call or a launch failed                */
    MA_ENOMEM = 4         /* the device workspace could not be allocated          */
} ma_status;

/*
 * monarch_attn_fwd -- O = M^(T) V for every (batch, head) slice.
 *
 * Operation: Sec. 3 of the paper; the T-step alternating maximisation
 * (eqs. R_update, L_update with beta_r, beta_l) from L^(0) = I, followed by
 * eq. monarch_multiply.  Organised as in the paper's Implementation paragraph
 * (state form, L and R kept on chip).
 *
 * q, k, v : DEVICE pointers to [B, H, N, d] row-major contiguous tensors of
 *           element type `dtype`, 16-byte aligned.  Read only.
 * out     : DEVICE pointer to a [B, H, N, d] tensor of the same type, 16-byte
 *           aligned, not overlapping q, k or v.  Fully overwritten.
 *           All four buffers are owned by the caller; the library neither
 *           frees nor retains them.
 * B, H    : batch and head counts (>= 0); B * H * max(m, b) < 2^31 (one
 *           workgroup per block or class of every head), else MA_EUNSUPPORTED.
 * N, m, b : sequence length, number of blocks and block size:
 *           m = ceil(N / b), i.e. (m - 1) * b < N <= m * b (m = 0 for an
 *           empty sequence, N = 0; b >= 1).  When N < m * b
 *           the sequence is post-padded to m * b rows as in Appendix
 *           "Padding and Masking": the padded rows of Q, K, V count as zero
 *           rows (they are not read), keys at positions >= N are masked out
 *           of every R softmax (omega = -inf on Z_R), and only the N real rows
 *           of out are written.  The padded query rows take part in the
 *           iteration like the others.  Supported: 1 <= m, b <= 128.
 * d       : head dimension; supported: d <= 128, a multiple of 8 (bf16,
 *           fp16) or 4 (fp32), so that every row is a whole number of 16-byte
 *           chunks.  The kernels work on tiles of width D = 64, 96 or 128
 *           (the smallest that holds d) with the extra columns zero.  fp32
 *           also needs tile(m)*D <= 8192 and tile(b)*D <= 8192, where
 *           tile(x) is the kernels' tile height for x rows: the smallest of
 *           16, 32, 64 and 128 that holds x.
 * T       : number of (R, L) update pairs, 1 <= T <= 64 for fp32 and
 *           1 <= T <= MONARCH_ATTN_MAX_T_16BIT for bf16 and fp16 (larger T:
 *           MA_EUNSUPPORTED).
 * dtype   : an ma_dtype value.
 * stream  : the hipStream_t to launch on (NULL = the null stream).
 *
 * Asynchronous on `stream`: returns after enqueueing, with no host
 * synchronisation.  A call with B, H or N zero has nothing to compute: once
 * the other arguments check out it returns MA_OK, launching nothing and
 * reading no pointer (they may be NULL); this holds for every entry point.
 * Arguments are checked before any HIP call; on MA_EINVAL or
 * MA_EUNSUPPORTED nothing is launched and `out` is untouched.  Path 1 (see
 * monarch_attn_set_path) uses a device workspace (3 m b d elements plus 2 m b
 * floats per head) owned by the library, one per (device, stream): calls on
 * different streams may run concurrently, and calls on one stream (from any
 * host thread) are enqueued one whole call at a time.  A stream's workspace
 * is grown with hipMalloc by the first call that needs more, after waiting
 * for that stream.  After the launches hipGetLastError is checked (MA_EHIP).
 *
 * HIP graph capture: a call on a stream being captured is recorded as its
 * kernel launches, with the stream's workspace address baked in.  It makes
 * no allocation, wait or event call, so the stream's workspace must already
 * be large enough (an earlier call of that size on the same stream);
 * otherwise the call fails with MA_EUNSUPPORTED and records nothing.  A
 * buffer that a captured call used is never freed when a later call grows
 * that workspace, only by monarch_attn_release_workspace, so captured graphs
 * stay valid until then.  The first call on that stream not under capture
 * after a capture moves the stream to a fresh buffer, so eager calls never
 * share one with a graph.  All graphs captured on one stream between two
 * eager calls share one buffer: such graphs must not be replayed at the
 * same time (on different streams) as each other.  Capture with per-launch timing enabled fails with
 * MA_EUNSUPPORTED.  The same holds for every entry point that takes a
 * stream.
 * The message of the last failure on the calling thread is returned by
 * monarch_attn_last_error().
 */
int monarch_attn_fwd(const void *q, const void *k, const void *v, void *out,
                     int64_t B, int64_t H, int64_t N, int64_t d,
                     int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

/*
 * monarch_attn_fwd_noalloc -- monarch_attn_fwd for callers that cannot
 * allocate device memory: code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc.  Same operation, arguments, kernels and
 * results (bit for bit) as monarch_attn_fwd, but the states of the half-step
 * path live in a scratch array that the library holds for the whole process
 * on every device it runs on (MONARCH_ATTN_NOALLOC_SCRATCH_BYTES per device,
 * set up by the first such call on that device), instead of the per-stream
 * workspace.  The call makes no hipMalloc, hipFree or other allocating call.
 *
 * A call whose states need more than MONARCH_ATTN_NOALLOC_SCRATCH_BYTES
 * (monarch_attn_workspace_bytes) returns MA_EUNSUPPORTED, launching nothing.
 * All calls on one device share its one scratch array, and the array keeps
 * the last call's contents: calls that can overlap on one device (different
 * streams, or replays of captured graphs on different streams) race and must
 * be ordered by the caller.  Nothing in the array needs to start at zero.
 */
int monarch_attn_fwd_noalloc(const void *q, const void *k, const void *v, void *out,
                             int64_t B, int64_t H, int64_t N, int64_t d,
                             int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

#define MONARCH_ATTN_NOALLOC_SCRATCH_BYTES (64ull << 20)

/*
 * monarch_attn_fwd_varlen -- monarch_attn_fwd over a batch of sequences of
 * different lengths, each post-padded to N rows (Appendix "Padding and
 * Masking", which names batched sequences padded to a maximum length as the
 * second use of its mask).
 *
 * lens : DEVICE pointer to B int32 values, 4-byte aligned, not overlapping
 *        out; lens[beta] is the number of real rows of batch element beta
 *        (for all its heads).  Read by the kernels, so its values are not
 *        checked on the host: they are clamped to 0..N.  Owned by the caller.
 * Batch element beta is computed as the single sequence of its first
 * lens[beta] rows, post-padded with zero rows to m * b at the batch's m and
 * b: rows >= lens[beta] of q, k, v count as zero whatever they hold (the
 * kernels may load them, up to row N - 1, and replace them by zero), keys at
 * positions >= lens[beta] are masked out of every R softmax, and the padded
 * query rows take part in the iteration as zero rows.  Here whole key blocks can be
 * padding, which the paper leaves undefined: such a block gets R = 0 and no
 * weight in the L softmax (Z_L = -inf), so that M keeps unit row sums and
 * zero columns at every padded key; a sequence of length 0 has M = 0.
 * Rows lens[beta]..N-1 of out are written as zero.  With lens[beta] = N for
 * every beta the result is that of monarch_attn_fwd.
 * The other arguments, the errors, the workspace and the asynchrony are
 * those of monarch_attn_fwd.
 */
int monarch_attn_fwd_varlen(const void *q, const void *k, const void *v, void *out, const int32_t *lens,
                            int64_t B, int64_t H, int64_t N, int64_t d,
                            int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

/*
 * monarch_attn_fwd_prepad -- monarch_attn_fwd over pre-padded sequences:
 * the padding rows come before the real ones (the last sentence of Appendix
 * "Padding and Masking": the key mask then removes the positions below
 * m b - n of the padded sequence, n its real rows, instead of those from n
 * on).
 *
 * lens : NULL, or a DEVICE pointer to B int32 values as in
 *        monarch_attn_fwd_varlen (4-byte aligned, clamped to 0..N).
 *        NULL: all N rows of every head are real, and the sequence is
 *        pre-padded with m b - N zero rows.  Otherwise batch element beta
 *        holds its lens[beta] real rows as the LAST lens[beta] of its N rows
 *        (a left-padded batch), pre-padded with zero rows to m b; rows
 *        0 .. N - lens[beta] - 1 of q, k, v count as zero whatever they hold
 *        and are written as zero in out.  Whole key blocks can then be
 *        padding, with the convention of monarch_attn_fwd_varlen (R = 0, no
 *        weight in the L softmax).
 * The result is that of the post-padded problem on the row-reversed tensors,
 * row-reversed: reversing the m b positions sends block l to m - 1 - l and
 * row j to b - 1 - j, which keeps L^(0) = I and both softmaxes.  The kernels
 * run exactly that, reading and writing rows in reverse order.  The other
 * arguments, the errors, the workspace and the asynchrony are those of
 * monarch_attn_fwd (paths 1 and 2 only; path 3 returns MA_EUNSUPPORTED).
 */
int monarch_attn_fwd_prepad(const void *q, const void *k, const void *v, void *out, const int32_t *lens,
                            int64_t B, int64_t H, int64_t N, int64_t d,
                            int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

/*
 * monarch_attn_fwd_objective -- monarch_attn_fwd, plus the value of the
 * variational objective f(M; Q, K) = <M, s Q K^T> + H(M) (Sec. 3, eq.
 * softmax_variational_attention, in its separable form for Monarch M) after
 * every step t = 1..T: a convergence diagnostic.  After the L update of step
 * t, f equals the sum over the query rows of the logsumexp of that update's
 * logits (the L update maximises f over L with R fixed, and row by row that
 * maximum is the logsumexp, eq. softmax_variational); the kernels form it
 * from the statistics of their softmax and reduce it in a fixed order, so
 * the result is deterministic.  When N < m * b the sum runs over the m * b
 * rows of the padded problem.  f never exceeds the exact-softmax value
 * sum_rows logsumexp(s q K^T).
 *
 * obj : DEVICE pointer to B*H*T floats, 4-byte aligned, not overlapping the
 *       tensors; obj[(b*H + h)*T + t - 1] receives f for (batch b, head h,
 *       step t).  Owned by the caller.
 * The other arguments, the errors and the asynchrony are those of
 * monarch_attn_fwd; the workspace also holds B*H*T*b floats of partial sums.
 */
int monarch_attn_fwd_objective(const void *q, const void *k, const void *v, void *out, float *obj,
                               int64_t B, int64_t H, int64_t N, int64_t d,
                               int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

/*
 * monarch_attn_exact_fwd -- exact softmax attention O = softmax(s Q K^T) V,
 * s = 1/sqrt(d) (eq. softmax_attention), the reference that the Monarch
 * output's quality is measured against, and the logsumexp of every row of
 * s Q K^T (natural log).  Their sum over the rows is the largest value the
 * objective of monarch_attn_fwd_objective can take (the exact softmax
 * maximises it, eq. softmax_variational_attention).
 *
 * q, k, v, out : DEVICE pointers to [B, H, N, d] tensors as in
 *                monarch_attn_fwd (any N >= 1 below 2^31; d as there;
 *                B * H * ceil(N / 64) < 2^31, else MA_EUNSUPPORTED).
 * lse          : NULL, or a DEVICE pointer to B*H*N floats (4-byte aligned,
 *                not overlapping the tensors), lse[(b*H + h)*N + row].
 * Asynchronous on `stream`; arguments are checked before any HIP call
 * (MA_EINVAL / MA_EUNSUPPORTED, nothing launched); uses no workspace.
 */
int monarch_attn_exact_fwd(const void *q, const void *k, const void *v, void *out, float *lse,
                           int64_t B, int64_t H, int64_t N, int64_t d, int32_t dtype, void *stream);

/*
 * monarch_attn_bwd -- the gradient of monarch_attn_fwd: given dout = dL/dO,
 * dq, dk, dv = dL/dQ, dL/dK, dL/dV of the same T-step computation (reverse
 * mode through the unrolled iteration of Sec. 3 from L^(0) = I and eq.
 * monarch_multiply, the factors entering through eqs. R_update and L_update
 * with beta_r, beta_l).  The paper states no gradient; this is the exact
 * derivative of the forward pass as defined there, including the entropy
 * terms c_L and the normalisers c_R, and the key mask of Appendix "Padding
 * and Masking" when N < m * b.  Padded rows receive no gradient (dq, dk, dv
 * have N rows).
 *
 * q, k, v, dout : DEVICE pointers to [B, H, N, d] tensors of element type
 *                 `dtype`, 16-byte aligned, read only.
 * dq, dk, dv    : DEVICE pointers to [B, H, N, d] tensors of that type,
 *                 16-byte aligned, overlapping neither each other nor the
 *                 inputs.  Fully overwritten.  All owned by the caller.
 * B, H, N, d, m, b, T, dtype, stream : as monarch_attn_fwd, and in addition
 *                 T <= 32 for fp32 and T <= MONARCH_ATTN_MAX_T_16BIT_BWD
 *                 for bf16 and fp16 (else MA_EUNSUPPORTED).
 *
 * Runs the forward half-steps again, keeping the states of every step, then
 * one launch per half-step in reverse order; all of it on `stream`,
 * asynchronously.  The arithmetic of the reverse sweep is fp32 (the states
 * of the recomputed forward pass are in the element type, as in
 * monarch_attn_fwd), and the result is deterministic (no atomics).
 * Workspace: monarch_attn_bwd_workspace_bytes(), in the same per-(device,
 * stream) buffer as monarch_attn_fwd (same rules).  Errors as
 * monarch_attn_fwd.
 */
int monarch_attn_bwd(const void *q, const void *k, const void *v, const void *dout,
                     void *dq, void *dk, void *dv,
                     int64_t B, int64_t H, int64_t N, int64_t d,
                     int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

/*
 * monarch_attn_bwd_varlen -- the gradient of monarch_attn_fwd_varlen (a batch
 * of sequences padded to N rows, lens[B] real rows per batch element, device
 * int32, clamped to 0..N; see there).  Key blocks of padding only have R = 0
 * and no L weight, so they pass no gradient.  Rows lens[beta]..N-1 of q, k,
 * v count as zero in the forward pass, so rows lens[beta]..N-1 of dq, dk and
 * dv are written as zero, and those rows of dout and of the inputs are
 * ignored whatever they hold.  lens must not overlap dq, dk or dv.  The
 * other arguments, the limits, the workspace and the errors are those of
 * monarch_attn_bwd.
 */
int monarch_attn_bwd_varlen(const void *q, const void *k, const void *v, const void *dout,
                            void *dq, void *dk, void *dv, const int32_t *lens,
                            int64_t B, int64_t H, int64_t N, int64_t d,
                            int64_t m, int64_t b, int32_t T, int32_t dtype, void *stream);

/* MA_OK if monarch_attn_bwd supports (N, d, m, b, T, dtype), else MA_EINVAL or
 * MA_EUNSUPPORTED (with last_error set).  Makes no HIP call. */
int monarch_attn_bwd_check(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype);

/* Bytes of device workspace monarch_attn_bwd needs (0 on bad arguments):
 * 2T state tensors of m b d elements and 2T - 1 arrays of m b floats per
 * head for the recomputed forward pass, 2 N d floats (dQ, dK accumulators),
 * 3 m b D floats (D = 64, 96 or 128, the smallest that holds d) and 2 m b floats
 * (state gradients) per head, each array rounded up to 256 bytes.  Makes no
 * HIP call. */
size_t monarch_attn_bwd_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d,
                                        int64_t m, int64_t b, int32_t T, int32_t dtype);

/* Text of the last failure on this thread ("" if none).  Valid until the next
 * call into the library from this thread. */
const char *monarch_attn_last_error(void);

/* Identifier of the sources the library was built from: the first 16 hex
 * digits of a SHA-256 over the kernel, dispatch and C ABI sources and this
 * header (paper_2505_18698_amd/build.py computes it).  A static string; makes
 * no HIP call.  The Python binding refuses a library whose identifier does
 * not match the sources beside it. */
const char *monarch_attn_build_id(void);

/* MA_OK if (N, d, m, b, T, dtype) is a supported shape, else MA_EINVAL or
 * MA_EUNSUPPORTED (with last_error set).  Makes no HIP call. */
int monarch_attn_check(int64_t N, int64_t d, int64_t m, int64_t b, int32_t T, int32_t dtype);

/* Bytes of device workspace monarch_attn_fwd needs for this shape (0 on bad
 * arguments).  Makes no HIP call. */
size_t monarch_attn_workspace_bytes(int64_t B, int64_t H, int64_t N, int64_t d,
                                    int64_t m, int64_t b, int32_t T, int32_t dtype);

/* Free the workspaces of the current device (all streams), including every
 * buffer kept alive for captured graphs (see monarch_attn_fwd): a graph that
 * captured a call must not be replayed after this.  Waits for calls being
 * enqueued and for the device to go idle first, so it may be called while
 * other threads use the library; their next call allocates again. */
int monarch_attn_release_workspace(void);

/*
 * Execution path of monarch_attn_fwd (process-wide; returns the previous
 * value, or -1 on an unknown value):
 *   0  automatic (default), see below;
 *   1  one launch per half-step (the state form of the paper's
 *      Implementation paragraph, the states crossing launches through the
 *      workspace);
 *   2  one workgroup per (batch, head) running every half-step with Q, K and
 *      all states in LDS (the fully fused one-head-per-block kernel for short
 *      sequences, Sec. 4, paragraph "Benchmarking"): bf16 or fp16, d <= 64,
 *      m <= 16 and b <= 16; any other shape returns MA_EUNSUPPORTED.  Uses
 *      no workspace.
 *   3  one workgroup per (batch, head, group of residue classes j) running
 *      every step in one launch with the states of its classes in LDS (the
 *      classes of a head are independent given K and V): bf16 or fp16,
 *      d <= 64, m <= 64 and b <= 32, in monarch_attn_fwd and
 *      monarch_attn_fwd_noalloc only (not with per-sequence lengths or the
 *      objective); any other call returns MA_EUNSUPPORTED.  Uses no
 *      workspace.
 * Automatic selection takes path 2 where it applies; else path 3 where it
 * applies with m <= 32; else path 1.  All paths compute the same operation with the same
 * per-unit arithmetic, and give the same bits.
 */
int monarch_attn_set_path(int32_t path);

/*
 * Per-launch timing, for measurement only.  While enabled (flag != 0), every
 * call of the library (forward, objective, exact attention, gradient) records
 * a HIP event before and after each kernel it launches, on the caller's
 * stream.  monarch_attn_timing_read() synchronises
 * on the last call's final event and writes, for at most `cap` launches of
 * that call, the duration in milliseconds to ms[i] and the kernel kind to
 * kind[i] (0 R half-step, 1 L half-step, 2 last R half-step with Y,
 * 3 last L half-step with the Monarch product and the store of O,
 * 4 the one-workgroup-per-head kernel, 5 the sum of the objective shares,
 * 6 exact attention, 7 an L half-step of the gradient, 8 an R half-step of
 * the gradient, 9 the one-workgroup-per-group-of-classes kernel); it returns
 * the number of launches of that call, or -1 on error.
 */
int monarch_attn_timing_enable(int32_t flag);
int32_t monarch_attn_timing_read(float *ms, int32_t *kind, int32_t cap);

#ifdef __cplusplus
}
#endif

#endif /* MONARCH_ATTN_H */
