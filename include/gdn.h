/*
 * gdn.h -- C ABI of the MI355X (gfx950) gated delta-rule library (libgdn.so).
 *
 * The operation (paper, section 2.2 "The model"; section 3.2 "A chunked
 * delta-rule scan for the recurrent layers"): every recurrent layer keeps one
 * state matrix per head, updated token by token.  With the state stored as
 * S in R^{dv x dk}, a scalar log-decay g_t per (token, head), alpha_t = exp(g_t),
 * and a write strength beta_t,
 *
 *     S_t = alpha_t S_{t-1} (I - beta_t k_t k_t^T) + beta_t v_t k_t^T
 *     o_t = S_t (scale q_t)                     (read after the update)
 *
 * gdn_chunk_prefill evaluates this over a whole prompt in the chunked
 * intra-/inter-chunk form of section 3.2 (chunks of `chunk` tokens: token-token
 * products, a forward-substituted unit-lower-triangular system, correction and
 * output products, and a short recurrence across chunks).  gdn_decode_step is
 * one token of the same recurrence for a batch of sequences.
 *
 * Conventions shared by every entry point
 *  - Every tensor pointer is a DEVICE pointer owned by the caller; the library
 *    keeps no reference after the call returns and allocates no device memory.
 *  - All tensors are contiguous and row-major.  Alignment: the prefill's q, k,
 *    v, o, S0, S_T and the decode state S start on 16-byte boundaries; every
 *    other pointer (g, beta, cu_seqlens, the decode step's q, k, v, o) only
 *    needs the alignment of its element type.
 *  - `io_dtype` selects the element type of q, k, v and o: GDN_F32 (float) or
 *    GDN_BF16 (bfloat16).  g, beta and the state are always fp32.
 *  - `stream` is a hipStream_t (NULL = the default stream).  Work is enqueued
 *    asynchronously; a kernel fault surfaces at the caller's next
 *    synchronisation, not in the returned status.
 *  - Errors are returned, never raised; nothing aborts.  Every argument check
 *    runs before the first HIP call, so an invalid call touches no device state.
 *    gdn_last_error_message() gives a thread-local description of the last
 *    failure on the calling thread.
 *  - Inputs and outputs must not overlap, except S0 == S_T (in place).
 */
#ifndef GDN_H
#define GDN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gdn_status {
    GDN_OK = 0,
    GDN_ERR_INVALID_ARG = 1,   /* null/misaligned pointer, bad size or dtype      */
    GDN_ERR_UNSUPPORTED = 2,   /* valid but not implemented (dk, dv, chunk)       */
    GDN_ERR_WORKSPACE = 3,     /* workspace missing or smaller than required      */
    GDN_ERR_HIP = 4,           /* a HIP launch/runtime call failed                */
    GDN_ERR_WAIT = 5           /* a bounded wait between the library's own
                                  workgroups gave up (gdn_workspace_status)       */
} gdn_status;

typedef enum gdn_dtype { GDN_F32 = 0, GDN_BF16 = 1 } gdn_dtype;

/* Bit flags of the _ex entry points: input transforms done inside the kernels,
   and at most one evaluation plan (none: the library chooses). */
typedef enum gdn_flags {
    GDN_QK_L2NORM = 1,         /* q and k scaled per (token, head) to k / sqrt(|k|^2 + 1e-6)          */
    GDN_GATE_LOGITS = 2,       /* g and beta arrive as logits a, b: g = -softplus(a), beta = sigmoid(b) */
    GDN_PLAN_SEQUENTIAL = 16,  /* one chain over every chunk of a sequence                             */
    GDN_PLAN_SEGMENTED = 32,   /* segment-parallel, narrow: one workgroup per 16 state rows             */
    GDN_PLAN_WIDE = 64,        /* segment-parallel, wide: a workgroup holds a whole state               */
    GDN_TEST_WITHHOLD = 256    /* test only: forces the failure path of the one-launch form's wait      */
} gdn_flags;

/* Library version, (major << 16) | minor. */
int gdn_version(void);

/* Static text for a status code ("GDN_OK", ...); "unknown status" otherwise. */
const char* gdn_status_string(int status);

/* Thread-local description of the last non-OK status on this thread ("" if none). */
const char* gdn_last_error_message(void);

/*
 * Status of the calls made with this workspace (its first 8 bytes), for the
 * one-launch form of the bf16 sequential prefill.  There the chunk-terms
 * workgroups publish each chunk's terms with a per-call tag and the chain
 * workgroups of the same launch wait for it, polling at most 2^22 times per
 * call (seconds).  The chunk-terms workgroups never wait and are dispatched
 * first, so the bound is reached only when they cannot run (the device held by
 * other work for that long).  A chain that gives up stores the call's tag in
 * the workspace's status word and writes NaN to the rest of its outputs and to
 * its final state; the call itself has already returned GDN_OK.
 *
 * This function waits for `stream` (NULL: the default stream), reads the word,
 * and returns GDN_ERR_WAIT if a call of this process on this workspace gave up
 * since the last check (and clears the word), else GDN_OK.  `workspace` NULL
 * checks the scratch of gdn_chunk_prefill_noalloc on the device of `stream`.
 * A workspace of fewer than 8 bytes (calls that needed none) is always GDN_OK.
 * GDN_ERR_HIP if a HIP call fails.  Not for use under graph capture.
 *
 * GDN_TEST_WITHHOLD (a flag of the _ex entry points, for tests of this path):
 * in the one-launch form the chunk-terms workgroups publish nothing and the
 * chain polls at most 1024 times, so every chain gives up, every kernel still
 * exits normally, the outputs are NaN and this function reports GDN_ERR_WAIT.
 * Calls that do not take the one-launch form ignore it.
 */
gdn_status gdn_workspace_status(const void* workspace, size_t workspace_bytes, void* stream);

/*
 * Workspace (device scratch, bytes) that gdn_chunk_prefill needs for these
 * sizes: the per-chunk state-independent terms of section 3.2 (decay prefix
 * sums, the inverse of the triangular system, the masked query-key product)
 * and, for ragged input, the sanitised sequence table.  Same argument meaning
 * as gdn_chunk_prefill (`n_seqs` = 0 for dense input).  Returns 0 for
 * arguments gdn_chunk_prefill would reject.  Pure host arithmetic.
 */
size_t gdn_chunk_prefill_workspace_bytes(int B, int T, int H, int dk, int dv, int chunk,
                                         int n_seqs, int io_dtype);

/*
 * Workspace for gdn_chunk_prefill_ex with this `flags` and `segments` (see the
 * plans below): the bytes the plan needs on a 256-CU device, and never less than
 * the sequential form's.  flags = segments = 0 is
 * gdn_chunk_prefill_workspace_bytes.  Returns 0 for arguments the prefill would
 * reject.  Pure host arithmetic.
 */
size_t gdn_chunk_prefill_workspace_bytes_ex(int B, int T, int H, int dk, int dv, int chunk,
                                            int n_seqs, int io_dtype, int flags, int segments);

/*
 * Chunked prefill (section 3.2).
 *
 * Dense input (cu_seqlens == NULL, n_seqs == 0): B independent sequences of T
 * tokens.  Ragged input (cu_seqlens != NULL): B must be 1 and the T tokens are
 * n_seqs packed sequences; cu_seqlens is a DEVICE int32 array [n_seqs + 1] with
 * cu[0] = 0, cu[i] <= cu[i+1], cu[n_seqs] = T.  Chunks restart at every
 * sequence start; a sequence of length 0 returns S_T = S0.  The contents of
 * cu_seqlens are not checked on the host; offsets outside that contract are
 * clamped on the device into a nondecreasing partition of [0, T] (no
 * out-of-bounds access), which is then what gets computed.
 *
 *   q, k     [B, T, H, dk]  io_dtype        keys are used as given (no renormalisation)
 *   v        [B, T, H, dv]  io_dtype
 *   g, beta  [B, T, H]      fp32            log-decay (alpha = exp g) and write strength
 *   S0       [n, H, dv, dk] fp32 or NULL    initial state (NULL = zeros); n = B or n_seqs
 *   o        [B, T, H, dv]  io_dtype        output (written)
 *   S_T      [n, H, dv, dk] fp32 or NULL    final state (written unless NULL; may == S0)
 *   dk, dv   64 or 128;  T >= 0;  B, H >= 1
 *   chunk    tokens per chunk: 64 runs the tuned kernels (every plan and
 *            snapshots); 16, 32 and 128 run a generic path (section 3.2 leaves the
 *            chunk length free; the result equals the recurrence at every length):
 *            per (chunk, head) the decay-masked products and the forward
 *            substitution in fp32, then one chain per (sequence, head, 16 state
 *            rows) on the vector units -- sequential plan only, no snapshots
 *            (GDN_ERR_UNSUPPORTED), workspace per (chunk slot, head) of
 *            16 chunk + 8 chunk^2 bytes; other lengths GDN_ERR_UNSUPPORTED
 *   scale    multiplies q (o_t = S_t (scale q_t)); 1.0f gives the plain rule
 *   workspace / workspace_bytes   device scratch of at least
 *            gdn_chunk_prefill_workspace_bytes(...) bytes, 256-byte aligned; its
 *            contents on entry are ignored, except its first 8 bytes (the
 *            status word of gdn_workspace_status), and on exit are unspecified.
 */
gdn_status gdn_chunk_prefill(const void* q, const void* k, const void* v,
                             const float* g, const float* beta, const float* S0,
                             void* o, float* S_T,
                             int B, int T, int H, int dk, int dv, int chunk,
                             const int32_t* cu_seqlens, int n_seqs,
                             int io_dtype, float scale,
                             void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * Chunked prefill with grouped key heads: q and k carry H_k heads and each of
 * the H value heads reads one of them, value head h the key head h / (H / H_k)
 * (section 2.2 keeps one state per value head; the model family's recurrent
 * layers share query and key heads across groups of value heads).  Every
 * value head still has its own state, gate g, write strength beta and output.
 *
 *   q, k     [B, T, H_k, dk] io_dtype
 *   v, o     [B, T, H, dv]   io_dtype
 *   g, beta  [B, T, H]       fp32
 *   S0, S_T  [n, H, dv, dk]  fp32 (as gdn_chunk_prefill)
 *   H_k      1 <= H_k <= H and H_k divides H (GDN_ERR_INVALID_ARG otherwise);
 *            H_k = H is gdn_chunk_prefill exactly
 * All other arguments, the workspace (gdn_chunk_prefill_workspace_bytes with the
 * value-head count H), the automatic plan and the errors are those of
 * gdn_chunk_prefill.
 */
gdn_status gdn_chunk_prefill_grouped(const void* q, const void* k, const void* v,
                                     const float* g, const float* beta, const float* S0,
                                     void* o, float* S_T,
                                     int B, int T, int H, int H_k, int dk, int dv, int chunk,
                                     const int32_t* cu_seqlens, int n_seqs,
                                     int io_dtype, float scale,
                                     void* workspace, size_t workspace_bytes,
                                     void* stream);

/*
 * Chunked prefill with the per-position input transforms done in its kernels
 * (section 3 batches the per-position operations around the projections over
 * the whole chunk; these are the ones that feed the scan) and a per-call
 * evaluation plan.  Arguments as gdn_chunk_prefill_grouped, plus:
 *   flags  0 or a combination of
 *          GDN_QK_L2NORM    q and k are taken as given and each row (token, key
 *                           head) is used scaled to x / sqrt(|x|^2 + 1e-6); `scale`
 *                           still multiplies q afterwards.  A zero row stays zero.
 *          GDN_GATE_LOGITS  the `g` and `beta` arguments hold logits a and b:
 *                           log-decay g = -softplus(a) = -log(1 + exp(a)), write
 *                           strength beta = 1 / (1 + exp(-b)).
 *          and at most one plan (none: the library chooses; results agree to
 *          rounding whichever plan runs).  Section 3.2: the chunk map is affine in
 *          the state, S_{c+1} = S_c M_c + N_c, so a sequence's chunks can be grouped
 *          into segments whose maps compose.
 *          GDN_PLAN_SEQUENTIAL  one chain walks every chunk of a sequence.
 *          GDN_PLAN_SEGMENTED   narrow segment-parallel form: dense input is cut
 *                           into segments; every segment's chain runs at once on the
 *                           values from a zero state (segment 0: from S0) and on zero
 *                           values from the identity (the segment's transition and
 *                           how the state entering it reaches its outputs); a scan
 *                           composes the entering states and a last pass adds each
 *                           segment's entering-state term to its outputs.  Ragged
 *                           input is never split (the plan is then sequential).
 *          GDN_PLAN_WIDE        wide segment-parallel form (dense bf16 input, dk ==
 *                           dv, without GDN_QK_L2NORM; GDN_ERR_UNSUPPORTED otherwise):
 *                           each workgroup holds a whole state of one head; the
 *                           segments' transitions (M_p, N_p) in one pass, a scan of
 *                           the entering states in near-fp32 precision, and a rerun
 *                           of every segment from its entering state with outputs.
 *          Other bits, or two plans: GDN_ERR_INVALID_ARG.
 *   segments  0: the plan's own count (the automatic plan chooses form and count
 *          from the compute units of the stream's device and the sizes);
 *          1: the sequential form; 2..64: that many segments per sequence (fewer
 *          when a sequence has fewer chunks), with GDN_PLAN_SEGMENTED or
 *          GDN_PLAN_WIDE only (GDN_ERR_INVALID_ARG otherwise, and outside 0..64).
 * A call whose workspace is too small for the split it would make uses fewer
 * segments, down to the sequential form.  flags = segments = 0 is
 * gdn_chunk_prefill_grouped.  The workspace:
 * gdn_chunk_prefill_workspace_bytes_ex(..., flags, segments).
 */
gdn_status gdn_chunk_prefill_ex(const void* q, const void* k, const void* v,
                                const float* g, const float* beta, const float* S0,
                                void* o, float* S_T,
                                int B, int T, int H, int H_k, int dk, int dv, int chunk,
                                const int32_t* cu_seqlens, int n_seqs,
                                int io_dtype, float scale, int flags, int segments,
                                void* workspace, size_t workspace_bytes,
                                void* stream);

/*
 * Bytes of device scratch that gdn_chunk_prefill_noalloc holds per device.
 */
#define GDN_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/*
 * gdn_chunk_prefill_ex without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  It calls no hipMalloc, hipFree or other
 * allocating routine: its scratch is a device array of GDN_NOALLOC_SCRATCH_BYTES
 * (64 MiB) inside the library, one per device, held from the library's first use
 * on that device until the process ends; its address is looked up on the first
 * call on each device (the device of `stream`, made current for the lookup).
 * Arguments, results, plans and errors as gdn_chunk_prefill_ex, with the plan
 * chosen for a workspace of GDN_NOALLOC_SCRATCH_BYTES; the caller still passes
 * every input and output.  Sizes whose sequential form needs more scratch than
 * that (gdn_chunk_prefill_workspace_bytes_ex(..., GDN_PLAN_SEQUENTIAL, 0) >
 * GDN_NOALLOC_SCRATCH_BYTES): GDN_ERR_WORKSPACE, nothing enqueued.  Nothing in
 * the scratch needs to start cleared.  Every call on one device shares that
 * device's scratch: calls that overlap in time on one device (different streams,
 * or host threads without ordering between their streams) race and give wrong
 * results; calls ordered on one stream are safe.
 */
gdn_status gdn_chunk_prefill_noalloc(const void* q, const void* k, const void* v,
                                     const float* g, const float* beta, const float* S0,
                                     void* o, float* S_T,
                                     int B, int T, int H, int H_k, int dk, int dv, int chunk,
                                     const int32_t* cu_seqlens, int n_seqs,
                                     int io_dtype, float scale, int flags, int segments,
                                     void* stream);

/*
 * The plan gdn_chunk_prefill_ex would take for these arguments, given a
 * workspace of `workspace_bytes` bytes and the compute units of the device of
 * `stream` (NULL: the current device): returns the segments per sequence (1 for
 * the sequential form, 0 for arguments the prefill would reject) and stores the
 * plan's GDN_PLAN_* bit in *form (when form is not NULL; 0 on rejection).
 * Queries the device's compute-unit count; enqueues nothing.
 */
int gdn_chunk_prefill_plan(int B, int T, int H, int dk, int dv, int n_seqs, int io_dtype, int flags,
                           int segments, size_t workspace_bytes, void* stream, int* form);

/*
 * Chunked prefill that also stores the state at chunk boundaries inside each
 * sequence: the hook for a cache of recurrent-state snapshots indexed by prompt
 * position (section 3, the engine's prefix-snapshot cache; section 6).  Arguments
 * as gdn_chunk_prefill, plus:
 *   snap_every  positive: a snapshot every snap_every chunks -- snapshot j
 *               (j = 1, 2, ...) of a sequence is its state after its first
 *               j * snap_every * chunk tokens, taken while that count is less than
 *               the sequence's length (the state at the end is S_T)
 *   snaps       [n, n_snap, H, dv, dk] fp32 DEVICE, n_snap = (T - 1) / (snap_every
 *               * chunk) (integer division; T bounds every sequence's length);
 *               snapshot j of sequence s at [s, j - 1]; entries past a sequence's
 *               last snapshot are left as they were.  16-byte aligned; may be NULL
 *               when n_snap is 0.  Must not overlap any other argument.
 * The sequential form always; the workspace is the one
 * gdn_chunk_prefill_workspace_bytes gives.  Errors as gdn_chunk_prefill, and
 * GDN_ERR_INVALID_ARG for snap_every < 1 or a missing or misaligned snaps.
 */
gdn_status gdn_chunk_prefill_snapshots(const void* q, const void* k, const void* v,
                                       const float* g, const float* beta, const float* S0,
                                       void* o, float* S_T,
                                       int B, int T, int H, int dk, int dv, int chunk,
                                       const int32_t* cu_seqlens, int n_seqs,
                                       int io_dtype, float scale,
                                       int snap_every, float* snaps,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/*
 * Snapshots with grouped key heads and the in-kernel input transforms: arguments
 * as gdn_chunk_prefill_snapshots plus H_k (as gdn_chunk_prefill_grouped; q and k
 * [B, T, H_k, dk]) and flags (as gdn_chunk_prefill_ex).  H_k = H and flags = 0
 * is gdn_chunk_prefill_snapshots.  The plan bits of `flags` are not accepted
 * (GDN_ERR_INVALID_ARG): snapshots always take the sequential form.
 */
gdn_status gdn_chunk_prefill_snapshots_ex(const void* q, const void* k, const void* v,
                                          const float* g, const float* beta, const float* S0,
                                          void* o, float* S_T,
                                          int B, int T, int H, int H_k, int dk, int dv, int chunk,
                                          const int32_t* cu_seqlens, int n_seqs,
                                          int io_dtype, float scale, int flags,
                                          int snap_every, float* snaps,
                                          void* workspace, size_t workspace_bytes,
                                          void* stream);

/*
 * One decode step (the recurrence at T = 1; section 2.2, section 3.2): one
 * token for each of B sequences.
 *
 *   q, k     [B, H, dk]        io_dtype
 *   v        [B, H, dv]        io_dtype
 *   g, beta  [B, H]            fp32
 *   S        [B, H, dv, dk]    fp32, read and updated IN PLACE
 *   o        [B, H, dv]        io_dtype, o = S_new (scale q)
 *   dk, dv   64 or 128;  B, H >= 1
 * Needs no workspace.
 */
gdn_status gdn_decode_step(const void* q, const void* k, const void* v,
                           const float* g, const float* beta, float* S, void* o,
                           int B, int H, int dk, int dv, int io_dtype, float scale,
                           void* stream);

/*
 * One decode step with grouped key heads (as gdn_chunk_prefill_grouped): q, k
 * [B, H_k, dk]; value head h reads key head h / (H / H_k).  v, o, g, beta and S
 * as gdn_decode_step; 1 <= H_k <= H and H_k divides H (GDN_ERR_INVALID_ARG
 * otherwise).  Needs no workspace.
 */
gdn_status gdn_decode_step_grouped(const void* q, const void* k, const void* v,
                                   const float* g, const float* beta, float* S, void* o,
                                   int B, int H, int H_k, int dk, int dv, int io_dtype, float scale,
                                   void* stream);

/*
 * One decode step with the input transforms of gdn_chunk_prefill_ex (`flags`)
 * done in its kernel; otherwise as gdn_decode_step_grouped.  Needs no workspace.
 */
gdn_status gdn_decode_step_ex(const void* q, const void* k, const void* v,
                              const float* g, const float* beta, float* S, void* o,
                              int B, int H, int H_k, int dk, int dv, int io_dtype, float scale,
                              int flags, void* stream);

/*
 * Causal softmax-attention prefill: the backbone's attention layers over a
 * prompt (section 5: the scores Q K^T of each head, a softmax over each query's
 * causal prefix, then the product with V; grouped query heads share a
 * key/value head).  Per sequence b, head h, query position i:
 *
 *     o_i = sum_{j <= i} softmax_j(scale q_i . k_j) v_j     (k, v of head h / (H / H_kv))
 *
 *   q, o   [B, T, H, d]     bf16 (io_dtype must be GDN_BF16)
 *   k, v   [B, T, H_kv, d]  bf16
 *   d      64 or 128;  1 <= H_kv <= H, H_kv divides H;  T >= 0 (T = 0: nothing to do)
 *   cu_seqlens, n_seqs   packed sequences as in gdn_chunk_prefill (B must be 1; DEVICE int32
 *          [n_seqs + 1]; each sequence attends only within itself; offsets outside the contract
 *          are clamped on the device into a nondecreasing partition of [0, T]), or NULL and 0
 *   scale  multiplies q . k (1 / sqrt(d) gives the usual attention)
 * The score matrix is never stored: the kernel keeps a running softmax per query
 * (fp32) and needs no workspace.  Errors: GDN_ERR_INVALID_ARG for bad sizes,
 * null or misaligned (16-byte) pointers or an unknown dtype; GDN_ERR_UNSUPPORTED
 * for GDN_F32 io or another d.
 */
gdn_status gdn_attention_prefill(const void* q, const void* k, const void* v, void* o,
                                 int B, int T, int H, int H_kv, int d,
                                 const int32_t* cu_seqlens, int n_seqs,
                                 int io_dtype, float scale, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GDN_H */
