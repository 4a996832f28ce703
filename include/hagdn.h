/*
 * hagdn.h -- C ABI of the MI355X (gfx950) chunkwise delta-rule prefill library.
 *
 * The operation (paper, Sec. 2.1 "Architecture of Linear-Attention Hybrids"
 * and "Chunkwise Map-Reduce-Map Execution"): prefill of a delta-rule
 * linear-attention layer.  Per sequence n and value head h a d_k x d_v state
 * is carried token by token; with S the state in d_v x d_k orientation,
 *
 *   Gated DeltaNet (GDN):  S_t = a_t S_{t-1} (I - b_t k_t k_t^T) + b_t v_t k_t^T
 *   KDA:                   S_t = S_{t-1} Diag(a_t) (I - b_t k_t k_t^T) + b_t v_t k_t^T
 *   output (both):         o_t = scale * S_t q_t       (reads the UPDATED state)
 *
 * where a_t = exp(g_t) is a scalar per (token, head) for GDN and a vector of
 * d_k per-key-channel decays for KDA.  The library computes this with the
 * chunkwise Map-Reduce-Map decomposition (chunk length 64, the paper's
 * setting in Sec. 7.1): operators #1-#4 (Gate, KKT, Solve, W/U) chunk-parallel,
 * operator #5 (H) sequential over chunks, operator #6 (O) chunk-parallel.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Pointers.  Every tensor pointer is a DEVICE pointer (HIP device memory of
 *   the current device), row-major, contiguous.  The caller owns every buffer,
 *   including the workspace.  The library never allocates or frees device
 *   memory, never synchronises the stream (except hagdn_device_status), and
 *   keeps no pointer after returning.  When T = 0 the token tensors (q, k, v,
 *   g, beta, o) are never read or written and may be NULL.
 * Layouts (T = T_total packed tokens, sequences delimited by cu_seqlens):
 *   q, k        [T, Hqk, Dk]   dtype
 *   v, o        [T, Hv,  Dv]   dtype
 *   g (GDN)     [T, Hv]        fp32 log-gate, a_t = exp(g) (g <= 0 expected)
 *   g (KDA)     [T, Hv, Dk]    fp32 per-key-channel log-gate
 *               Every finite g <= 0 is supported, i.e. every gate a in (0, 1]:
 *               KDA's factored decay switches, per 16-token block, to an exact
 *               form when some channel decays by more than e^40 over half a
 *               block (paper Sec. 2.1, the KDA variant).  g = -inf (a = 0) or
 *               NaN propagates NaN into the affected chunk's outputs.
 *   beta        [T, Hv]        fp32 write strength
 *   s0, s_final [N, Hv, Dk, Dv] fp32, the state stored as S^T (row = key
 *               channel, d_v contiguous).  s0 == NULL means a zero initial
 *               state; s_final == NULL skips writing the final state.
 *               s_final may alias s0 exactly (in-place update, on every
 *               path: the segmented path reads s0 only in a launch before
 *               the one that writes s_final); no other aliasing between
 *               arguments is allowed.
 *   cu_seqlens  [N+1] int32, DEVICE memory: cu[0] = 0, cu[N] = T,
 *               nondecreasing.  Zero-length sequences are allowed.  Chunks
 *               restart at every sequence start; no chunk spans two sequences.
 * Grouped heads: value head h reads q/k head h / (Hv / Hqk).
 * Supported shapes: Dk, Dv in {64, 128}; Hv % Hqk == 0; N >= 1; T >= 0.
 * dtype: HAGDN_BF16 (q/k/v/o bf16; fp32 state and accumulation, bf16
 *   intermediates) or HAGDN_F32 (everything fp32).
 * Alignment: q, k, v, o, s0, s_final and workspace 16-byte aligned; g, beta
 *   and cu_seqlens 4-byte aligned.
 * stream: a hipStream_t passed as void* (NULL = the default stream).  Work is
 *   enqueued asynchronously in stream order.
 * Errors: every entry point returns a hagdn_status.  Arguments are checked on
 *   the host before anything is enqueued; on a non-OK return nothing was
 *   launched (except HAGDN_EHIP: a launch failed) and hagdn_last_error()
 *   describes the problem.  Contents of cu_seqlens live on the device and are
 *   checked on the device (by the first kernel, or for N = 1 by the state
 *   kernel): if they are malformed, no token is processed (o is left
 *   untouched, s_final receives s0 or zeros) and hagdn_device_status()
 *   reports HAGDN_DEV_BAD_SEQLENS afterwards.
 */
#ifndef HAGDN_H
#define HAGDN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HAGDN_OK = 0,
  HAGDN_EINVAL = 1,        /* NULL required pointer, bad count, misalignment */
  HAGDN_EUNSUPPORTED = 2,  /* head dim / dtype outside the supported set     */
  HAGDN_EWORKSPACE = 3,    /* workspace smaller than *_workspace_size()      */
  HAGDN_EHIP = 4           /* a HIP runtime call or kernel launch failed     */
} hagdn_status;

typedef enum { HAGDN_F32 = 0, HAGDN_BF16 = 1 } hagdn_dtype;

/* Device-side status word written by every prefill call (by its first
 * kernel, or for a single sequence by its state kernel or, in an overlapped
 * call, by the setup kernel).  HAGDN_DEV_WAIT_TIMEOUT: in an overlapped call
 * (hagdn_set_overlap) a walk stopped waiting, after about a second, for a chunk
 * that its XCD's chunk-local work never published; the outputs are invalid.
 * Not expected: it would take a dispatch that leaves some XCD without the
 * workgroups of its queue (see hagdn_set_overlap). */
typedef enum {
  HAGDN_DEV_OK = 0,
  HAGDN_DEV_BAD_SEQLENS = 1,
  HAGDN_DEV_WAIT_TIMEOUT = 2
} hagdn_device_code;

/* Bytes of device workspace gdn_prefill needs for these sizes (0 if the
 * arguments are invalid; hagdn_last_error() then says why).  The workspace
 * holds the chunk and segment tables and the chunk-local factors of operators
 * #2-#6 (the state-independent parts of the per-chunk state update and output,
 * after Sec. 5's GEMM-first regrouping): Dk*Dk + Dk*Dv + 64*(Dk+Dv) elements
 * plus Dk floats per (chunk, value head) for chunks bounded by T/64 + N.  When
 * a sequence can span more than one segment of the state chain (Sec. 4's
 * Chunk-Seg-Seg mapping; see hagdn_segment_chunks) it also holds one segment
 * map, Dk*Dk elements plus Dk*Dv floats, per (segment, value head) for
 * segments bounded by (T/64 + N) / L + N, and a copy of s0 (Dk*Dv floats
 * per sequence and value head).  It always holds 2 KiB plus 4 bytes per
 * (chunk, value head) for the queues and ready flags of the overlapped
 * launch (hagdn_set_overlap).  The size depends on the segment length L in
 * force (hagdn_set_segment_chunks) and on the current device's compute units
 * (see hagdn_segment_chunks): query it after setting, with the device the
 * call will run on current. */
size_t gdn_prefill_workspace_size(int N, int T_total, int Hqk, int Hv, int Dk,
                                  int Dv, int dtype);

/* Gated DeltaNet prefill (scalar log-gate per token and value head).
 * Computes o [T, Hv, Dv] and, if s_final != NULL, the final states. */
int gdn_prefill(const void *q, const void *k, const void *v, const float *g,
                const float *beta, const float *s0, const int32_t *cu_seqlens,
                int N, int T_total, int Hqk, int Hv, int Dk, int Dv,
                float scale, int dtype, void *o, float *s_final,
                void *workspace, size_t workspace_bytes, void *stream);

/* Workspace bytes for kda_prefill (same meaning as above). */
size_t kda_prefill_workspace_size(int N, int T_total, int Hqk, int Hv, int Dk,
                                  int Dv, int dtype);

/* KDA prefill: as gdn_prefill, but g is the per-key-channel log-gate
 * [T, Hv, Dk]; the decay Diag(exp(g_t)) acts on the key side of the state
 * before the delta update. */
int kda_prefill(const void *q, const void *k, const void *v, const float *g,
                const float *beta, const float *s0, const int32_t *cu_seqlens,
                int N, int T_total, int Hqk, int Hv, int Dk, int Dv,
                float scale, int dtype, void *o, float *s_final,
                void *workspace, size_t workspace_bytes, void *stream);

/* Preprocessing flags (bit mask) for gdn_prefill_ex, kda_prefill_ex and the
 * decode entry points.  They fold the elementwise maps that turn a layer's raw
 * projections into the recurrence's inputs into the kernels' loads, so the
 * caller makes no separate pass over q, k, g and beta (the paper fuses the
 * layer's projection-side work around the LA core, Sec. 7 "Implementation
 * and Evaluation", full-layer implementation).  Each flag changes what the
 * corresponding argument holds:
 *   HAGDN_PRE_QK_L2NORM      q and k are raw: every token's q and k vector (per
 *                            q/k head) is divided by max(||x||_2, 1e-6) in fp32
 *                            before use (bf16: the result is rounded to bf16
 *                            where it is an MFMA operand);
 *   HAGDN_PRE_GATE_SOFTPLUS  g holds raw values x; the log-gate is -softplus(x)
 *                            = -log(1 + e^x), computed in fp32;
 *   HAGDN_PRE_BETA_SIGMOID   beta holds raw values x; the write strength is
 *                            1 / (1 + e^-x), computed in fp32.
 * Any other bit is rejected with HAGDN_EINVAL. */
typedef enum {
  HAGDN_PRE_QK_L2NORM = 1,
  HAGDN_PRE_GATE_SOFTPLUS = 2,
  HAGDN_PRE_BETA_SIGMOID = 4
} hagdn_pre_flags;

/* gdn_prefill / kda_prefill with preprocessing flags `pre` (a mask of
 * hagdn_pre_flags; 0 gives exactly gdn_prefill / kda_prefill).  Same
 * workspace size as without flags. */
int gdn_prefill_ex(const void *q, const void *k, const void *v, const float *g,
                   const float *beta, const float *s0, const int32_t *cu_seqlens,
                   int N, int T_total, int Hqk, int Hv, int Dk, int Dv,
                   float scale, int dtype, int pre, void *o, float *s_final,
                   void *workspace, size_t workspace_bytes, void *stream);
int kda_prefill_ex(const void *q, const void *k, const void *v, const float *g,
                   const float *beta, const float *s0, const int32_t *cu_seqlens,
                   int N, int T_total, int Hqk, int Hv, int Dk, int Dv,
                   float scale, int dtype, int pre, void *o, float *s_final,
                   void *workspace, size_t workspace_bytes, void *stream);

/* One decode step: a single new token for each of N sequences, advanced by
 * the token-by-token recurrence (paper Sec. 2.1, which notes that the
 * recurrent form serves decoding; Sec. 7.3 leaves decode to the serving
 * backend).  Starting from the state a prefill left in s_final, repeated
 * calls continue the sequence exactly as a longer prefill would (up to
 * rounding).
 *   q, k   [N, Hqk, Dk] dtype        v, o  [N, Hv, Dv] dtype
 *   g      GDN [N, Hv] / KDA [N, Hv, Dk] fp32 log-gate     beta [N, Hv] fp32
 *   state  [num_slots, Hv, Dk, Dv] fp32, a pool of states in the s_final
 *          layout, read and UPDATED IN PLACE
 *   slots  [N] int32 DEVICE memory, or NULL: sequence n uses pool slot
 *          slots[n] (NULL: slot n, and num_slots is taken as N).  A slot
 *          outside [0, num_slots) marks a padding entry: its output row is
 *          written as zeros and no state is touched.  Two live entries must
 *          not name the same slot (their updates would race).
 *   pre    preprocessing flags (hagdn_pre_flags).
 * No workspace.  N = 0 is a no-op.  Alignment: q, k, v, o and state
 * 16-byte aligned; g, beta, slots 4-byte aligned.  Returns a hagdn_status;
 * on a non-OK return nothing was launched (except HAGDN_EHIP). */
int gdn_decode(const void *q, const void *k, const void *v, const float *g,
               const float *beta, float *state, const int32_t *slots,
               int num_slots, int N, int Hqk, int Hv, int Dk, int Dv,
               float scale, int dtype, int pre, void *o, void *stream);
int kda_decode(const void *q, const void *k, const void *v, const float *g,
               const float *beta, float *state, const int32_t *slots,
               int num_slots, int N, int Hqk, int Hv, int Dk, int Dv,
               float scale, int dtype, int pre, void *o, void *stream);

/* Message for the last non-OK return on this host thread ("" if none). */
const char *hagdn_last_error(void);

/* Reads the device status word that the most recent call using this
 * workspace wrote.  Synchronises `stream`.  *code receives a
 * hagdn_device_code.  Returns HAGDN_OK, HAGDN_EINVAL or HAGDN_EHIP. */
int hagdn_device_status(const void *workspace, size_t workspace_bytes,
                        void *stream, int *code);

/* Per-kernel timing with HIP events recorded on the call's stream around each
 * kernel of every prefill and decode call made on this host thread between
 * begin and end (at most max_calls calls are recorded; later calls run
 * untimed).  hagdn_profile_end synchronises the recorded events and writes,
 * for each kernel i < min(max_kernels, hagdn_kernel_count()), its mean
 * duration in milliseconds over the calls that launched it into mean_ms[i]
 * (0 if none did); *calls receives the number of calls timed.  Returns a
 * hagdn_status. */
int hagdn_profile_begin(int max_calls);
int hagdn_profile_end(double *mean_ms, int max_kernels, int *calls);
int hagdn_kernel_count(void);
const char *hagdn_kernel_name(int i);

/* Library version: major * 10000 + minor * 100 + patch. */
int hagdn_version(void);

/* Segment length L of the state chain, in 64-token chunks (Sec. 4's
 * Chunk-Seg-Seg mapping).  Each sequence's chunks are cut into segments of L;
 * the composed affine map of every segment but the last is computed in
 * parallel, then each segment walks its own chunks from the state the earlier
 * segments' maps give.  Results are the same for every L up to rounding
 * order.  hagdn_set_segment_chunks(0) restores the automatic choice (a
 * function of N, T_total, Hv, Dv and the gate kind); a positive value forces
 * L for every later call in the process (both capped; see
 * hagdn_segment_chunks).  Not synchronised with calls in flight on other host
 * threads: set it before querying workspace sizes.  Returns HAGDN_OK or
 * HAGDN_EINVAL (chunks < 0 or > 2^20). */
int hagdn_set_segment_chunks(int chunks);

/* L that a call with these sizes and dtype would use now on the current
 * device (kda: 0 for gdn_prefill, 1 for kda_prefill); -1 on invalid sizes or
 * dtype.  The automatic choice depends on the device's compute-unit count
 * (queried once per device; the prefill calls use the same query).  On a host
 * where no HIP device can be queried, this and the workspace-size queries
 * answer for a 256-CU MI355X.  Automatic or forced, L is capped at the
 * largest value with 64 L Hv Dv elements of dtype below 2 GiB, so the output
 * rows of one segment stay addressable with 32-bit byte offsets; the cap
 * depends on Hv, Dv and dtype, never on T_total.  A call whose sequences can
 * be longer than L chunks takes the segmented path. */
int hagdn_segment_chunks(int N, int T_total, int Hv, int Dv, int dtype, int kda);

/* The same rule for a device of `cus` compute units (no device query): host
 * logic only.  -1 on invalid arguments (cus < 1 included). */
int hagdn_segment_chunks_for(int N, int T_total, int Hv, int Dv, int dtype, int kda, int cus);

/* Overlapped launch.  The state walk of chunk c needs only chunks 0..c's
 * chunk-local factors, so a call whose chains are walked whole (no segment
 * maps: see hagdn_segment_chunks) can run the chunk-local work (operators
 * #1-#4 and the state-independent factors of #5-#6) and the walks (#5 fused
 * with #6) in ONE launch: walk workgroups wait, chunk by chunk, for ready flags
 * that the chunk-local workgroups set once a block's factors are stored,
 * instead of for the whole chunk-local kernel (Sec. 4's cross-operator fusion,
 * with the Map of later chunks running beside the Reduce of earlier ones).
 * Each workgroup reads the id of the XCD it runs on and takes its work from
 * that XCD's queues: value heads h = x (mod 8) are produced and walked on XCD
 * x, so the factors and flags pass through one L2 (the L2s of different XCDs
 * are not coherent within a kernel).  It can run for GDN calls in bf16 with
 * Dk = Dv = 128 on devices of at least 256 CUs (8 XCDs) whose walks (N x Hv x
 * Dv/16 workgroups) fit in half the CUs.  It pays only when the chunk-local
 * work needs more than one round of the standalone kernel (more than 3 x CUs
 * (chunk, value head) blocks): mode 1, the default, uses it exactly then;
 * mode 2 wherever it can run (for tests and measurements); mode 0 never.
 * Results are bit-identical either way.  A tiny setup kernel clears the
 * queues and flags first (in the workspace).  Applies to every later call in
 * the process.  Returns HAGDN_OK or HAGDN_EINVAL. */
int hagdn_set_overlap(int mode);

/* 1 if a call with these sizes (kda: 0 gdn, 1 kda) would take the overlapped
 * launch on a device of `cus` compute units in the mode set now, 0 if not, -1
 * on invalid arguments.  Host logic only. */
int hagdn_overlap_for(int N, int T_total, int Hv, int Dk, int Dv, int dtype, int kda, int cus);

/* Allocation-free prefill, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): gdn_prefill_ex (kda = 0) or kda_prefill_ex (kda = 1) with the
 * same arguments except the workspace, which is a static device array of
 * hagdn_prefill_noalloc_capacity() bytes (128 MiB) that the library holds on
 * each device it runs on until the process ends.  The caller still provides
 * every input and output.  A call whose workspace (the *_workspace_size of
 * its sizes) exceeds the capacity returns HAGDN_EWORKSPACE before anything is
 * enqueued: 128 MiB covers, e.g., one 4096-token sequence at 16 value heads of
 * d = 128 (bf16: 98 MiB; about 1,330 (chunk, value head) blocks at d = 128).
 * Nothing is allocated or freed: no hipMalloc, hipFree or allocating library
 * call.  All calls on one device share the one array, so calls that overlap
 * in time on a device (other streams, other host threads) race and must be
 * serialised by the caller; calls in one stream are ordered.  Nothing in the
 * array needs to start at zero: every region is written before it is read.
 * The device status word of hagdn_device_status is not readable for these
 * calls.  Returns a hagdn_status. */
int hagdn_prefill_noalloc(int kda, const void *q, const void *k, const void *v, const float *g,
                          const float *beta, const float *s0, const int32_t *cu_seqlens, int N,
                          int T_total, int Hqk, int Hv, int Dk, int Dv, float scale, int dtype,
                          int pre, void *o, float *s_final, void *stream);
size_t hagdn_prefill_noalloc_capacity(void);

/* Measurement aids (no prefill or decode call uses them): the ceilings that
 * roofline fractions can be quoted against, measured on the current device.
 *   hagdn_measure_copy  enqueues one streaming copy of `bytes` (a multiple of
 *       16; src, dst 16-byte aligned device buffers that do not overlap) on 8
 *       workgroups per CU with nontemporal 16-byte accesses: time it with
 *       events on `stream` for the HBM bandwidth a plain kernel reaches.
 *   hagdn_measure_mfma  enqueues 4 x CUs workgroups of four waves, each wave
 *       running `iterations` rounds (1 .. 2^24) of 8 independent
 *       v_mfma_f32_16x16x32_bf16 chains; *flops receives the launch's floating
 *       point operations (2 per multiply-add).  sink (device, >= 16 x CUs
 *       floats) receives one value per wave.
 * Both return a hagdn_status. */
int hagdn_measure_copy(const void *src, void *dst, size_t bytes, void *stream);
int hagdn_measure_mfma(int iterations, float *sink, size_t sink_floats, double *flops, void *stream);

/* Debugging: where a prefill call with these sizes (kda: 0 gdn_prefill, 1
 * kda_prefill) keeps its chunk-local factors inside the workspace, so that a
 * test can read them after the call (they stay there until the workspace is
 * reused).  *offset receives the region's byte offset from the workspace
 * start and *bytes its size (padding included).  Per (chunk c, value head h)
 * block blk = c * Hv + h, with chunk c of a single sequence covering tokens
 * [64c, 64c + 64) (a batch: the chunks of sequence 0, then of sequence 1, ...),
 * Kt = (K * e^(gamma_last - gamma))^T, W and U~ operators #4 and P the
 * masked Q K^T of operator #2 (paper Sec. 2.1):
 *   HAGDN_WS_NM     -Kt W        Dk x Dk elements of dtype per block
 *   HAGDN_WS_B      Kt U~        Dk x Dv elements of dtype
 *   HAGDN_WS_QP     Q e^gamma - P W   64 x Dk elements of dtype
 *   HAGDN_WS_OLOC   P U~         64 x Dv elements of dtype
 *   HAGDN_WS_DECAY  e^gamma_last Dk floats (GDN: the first only)
 *   HAGDN_WS_SEG_A, HAGDN_WS_SEG_B  the segment maps (segmented calls only)
 * in the MFMA fragment orders that the walk kernels read: NM and Q' as 16 x 32
 * operand blocks of 64 lanes x 8 elements (lane = column + 16 x lane group,
 * element j of lane group g holding k index 4g + j (j < 4) or 12 + 4g + j),
 * B and O_loc lane-major per 16-column state tile with the tile's columns
 * interleaved in pairs of tiles (csrc/prefill.h gives the exact maps).
 * Returns HAGDN_OK or HAGDN_EINVAL.  Depends on the device like the
 * workspace size. */
typedef enum {
  HAGDN_WS_NM = 0,
  HAGDN_WS_B = 1,
  HAGDN_WS_QP = 2,
  HAGDN_WS_OLOC = 3,
  HAGDN_WS_DECAY = 4,
  HAGDN_WS_SEG_A = 5,
  HAGDN_WS_SEG_B = 6
} hagdn_ws_region;
int hagdn_workspace_region(int kda, int N, int T_total, int Hqk, int Hv, int Dk, int Dv, int dtype,
                           int region, size_t *offset, size_t *bytes);

#ifdef __cplusplus
}
#endif

#endif /* HAGDN_H */
