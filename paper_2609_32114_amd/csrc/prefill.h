// prefill.h -- internal interface between the host launcher (api.cpp) and the
// HIP kernels.  Not part of the public ABI (that is include/hagdn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hagdn {

constexpr int kChunk = 64;  // chunk length C (paper Sec. 7.1 uses C = 64)

// Preprocessing flags (the ABI's HAGDN_PRE_*): maps applied to the raw
// projections as the kernels load them.
constexpr int kPreQkNorm = 1;        // q, k <- x / max(||x||_2, 1e-6) per token and head
constexpr int kPreGateSoftplus = 2;  // g <- -softplus(g)
constexpr int kPreBetaSigmoid = 4;   // beta <- sigmoid(beta)
constexpr int kPreAll = 7;

// Everything one prefill call needs, resolved to device pointers.  The
// workspace regions are carved by api.cpp; per (chunk, value head) block
// `blk = chunk * Hv + h` each region holds one fixed-size block.  With
// Kt = (K * e^(gamma_last - gamma))^T, D = Diag(e^gamma_last) and W, U~, P
// the chunk-local operators #2-#4 (see k1_chunk_local.hip):
//   NM  -M = -(Kt W)                 (Dk x Dk: d_k out x d_k in)
//   Bc  B = Kt U~                    (Dk x Dv)
//   dec e^gamma_last                 (Dk floats; GDN: element 0 only)
//   Qp  Q' = Q * e^gamma - P W       (64 x Dk)
//   Ol  O_loc = P U~                 (64 x Dv)
// so that  S^T_{c+1} = D S^T_c + NM S^T_c + B  and  O = scale (Q' S^T_c + O_loc).
// NM and Qp are stored in fragment order (device.h): one 16-lane by 32 operand
// block after another, 64 lanes x 8 elements each; Bc and Ol lane-major, each
// lane's accumulator values of one state tile contiguous, so every consumer
// moves them with 16-byte lane accesses:
//   NM  operand blocks (row tile t of d_k out, k-block kb of d_k in), t-major;
//       slot j of lane (col, grp) = NM[16t + col][32kb + kmap(grp, j)]
//   Bc  per state tile n (d_v columns dv_of(n, 0..15), device.h), lane-major:
//       element (m, e) of lane (col, grp), at ((n*64 + lane)*(Dk/16) + m)*4 + e,
//       = B[16m + 4grp + e][dv_of(n, col)]
//   Qp  operand blocks (token tile nt, k-block kb of d_k), nt-major;
//       slot j of lane (col, grp) = Q'[16nt + col][32kb + kmap(grp, j)]
//   Ol  per state tile m, lane-major: element (nt, e) of lane (col, grp), at
//       ((m*64 + lane)*4 + nt)*4 + e, = O_loc[16nt + col][dv_of(m, 4grp + e)]
// Element type of every block is the I/O dtype (bf16 or fp32), dec is fp32.
//
// Segments (paper Sec. 4, the Chunk-Seg-Seg mapping): each sequence is cut into segments
// of seg_chunks chunks (the last may be shorter; an empty sequence still has
// one empty segment).  Composing the affine chunk maps over segment s gives
// its segment map  S^T_out = A_s S^T_in + B_s  (d_k x d_k, d_k x d_v), per
// (segment, value head) block:
//   Aseg  A_s in NM's fragment order and element type
//   Bseg  B_s fp32, in Bc's accumulator-block order
// Only segments followed by another segment of the same sequence have one.
// The first segment of a sequence has no A: its B walk starts from the
// initial state, so its B_s is the state entering the second segment, and
// no later segment reads s0.  That walk also copies s0 to s0c, where the first
// segment's state walk reads it: s_final may alias s0, and the last segment
// writes s_final in the same launch in which the first one starts.
struct PrefillArgs {
  const void *q, *k, *v;
  const float *g, *beta, *s0;
  const int32_t *cu_seqlens;
  int N, T, Hqk, Hv, Dk, Dv;
  int max_chunks;  // upper bound on chunks: T / 64 + N
  float scale;
  int pre;         // preprocessing flags (kPre*)
  void *o;
  float *s_final;
  // workspace
  int *status;         // [1] device status word (hagdn_device_code)
  int4 *seq_info;      // [N]  {first chunk, number of chunks, start token, length}
  int4 *chunk_info;    // [max_chunks] {sequence, start token, length, 0}; length 0 = unused
  void *NM, *Bc, *Qp, *Ol;
  float *dec;
  int seg_chunks;      // chunks per segment (>= 1)
  int max_segs;        // upper bound on segments: max_chunks / seg_chunks + N
  int2 *seq_seg;       // [N] {first segment, number of segments}
  int4 *seg_info;      // [max_segs] {sequence (-1 = unused), first chunk, chunks, index in sequence}
  void *Aseg;
  float *Bseg;
  float *s0c;          // [N, Hv, Dk, Dv] copy of s0 for sequences of several segments
  // 1: a single sequence, and no chunk index kernel ran: the kernels derive
  // the tables below from T and cu_seqlens (seq_info_at and friends)
  int single;
  int cus;             // compute units of the device the call runs on
  // Overlapped launch (the chunk-local work and the whole-chain walks in one
  // grid, launch_overlapped): workgroups [0, ovl_walk_wgs) walk, the rest run
  // chunk-local items.  ovl holds, per XCD x, a chunk-local item queue at
  // kOvlLocalQ + kOvlStride x and a walk tile queue at kOvlWalkQ + kOvlStride x
  // (each in its own 128-byte line), then a ready flag per (chunk, value head)
  // block at kOvlFlags + blk.  All zero before the launch (overlap_setup).
  int *ovl;
  int ovl_walk_wgs;
};

// XCDs of an MI355X.  Each has its own L2; the L2s are not coherent with each
// other within a kernel.
constexpr int kXcdCount = 8;
constexpr int kOvlStride = 32;                           // ints: one 128-byte line per queue
constexpr int kOvlLocalQ = 0;
constexpr int kOvlWalkQ = kXcdCount * kOvlStride;
constexpr int kOvlFlags = 2 * kXcdCount * kOvlStride;     // 2 KiB in
// Device status codes (hagdn_device_code).
constexpr int kDevBadSeqlens = 1;
constexpr int kDevWaitTimeout = 2;

// Id of the XCD the calling wave runs on.
__device__ __forceinline__ int xcc_id() {
  int x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & (kXcdCount - 1);
}
// Value heads served by XCD x in an overlapped launch: h = x, x + 8, ...
__host__ __device__ __forceinline__ int ovl_heads(int Hv, int x) { return Hv > x ? (Hv - x + kXcdCount - 1) / kXcdCount : 0; }

// The tables of the chunk index kernel, or for a single sequence (SINGLE:
// the kernels' separate instances for N = 1) the same entries derived in
// place.  A single sequence's cu_seqlens must be {0, T}; otherwise it has no
// chunks (nothing is written to o and its final state is the initial one)
// and the state kernels report HAGDN_DEV_BAD_SEQLENS.
__device__ __forceinline__ bool single_ok(const PrefillArgs &a) {
  return a.cu_seqlens[0] == 0 && a.cu_seqlens[1] == a.T;
}
// {first chunk, chunks, start token, length} of sequence n
template <bool SINGLE>
__device__ __forceinline__ int4 seq_info_at(const PrefillArgs &a, int n) {
  if constexpr (SINGLE) {
    const bool ok = single_ok(a);
    return make_int4(0, ok ? (a.T + kChunk - 1) / kChunk : 0, 0, ok ? a.T : 0);
  } else {
    return a.seq_info[n];
  }
}
// {first segment, segments} of sequence n
template <bool SINGLE>
__device__ __forceinline__ int2 seq_seg_at(const PrefillArgs &a, int n) {
  if constexpr (SINGLE) {
    const int nch = seq_info_at<true>(a, 0).y;
    return make_int2(0, nch > 0 ? (nch + a.seg_chunks - 1) / a.seg_chunks : 1);
  } else {
    return a.seq_seg[n];
  }
}
// {sequence (-1 = unused), first chunk, chunks, index in sequence} of segment s
template <bool SINGLE>
__device__ __forceinline__ int4 seg_info_at(const PrefillArgs &a, int s) {
  if constexpr (SINGLE) {
    const int nch = seq_info_at<true>(a, 0).y;
    const int nseg = nch > 0 ? (nch + a.seg_chunks - 1) / a.seg_chunks : 1;
    if (s >= nseg) return make_int4(-1, 0, 0, 0);
    const int c0 = s * a.seg_chunks;
    return make_int4(0, c0, min(a.seg_chunks, nch - c0), s);
  } else {
    return a.seg_info[s];
  }
}
// The device status word, written by one thread of the state kernel when the
// chunk index kernel did not run (a single sequence).
template <bool SINGLE>
__device__ __forceinline__ void single_status(const PrefillArgs &a) {
  if constexpr (SINGLE) {
    if (blockIdx.x == 0 && threadIdx.x == 0) a.status[0] = single_ok(a) ? 0 : 1;
  }
}

// One decode step: a single token for each of N sequences whose states live
// in a pool of num_slots states, sequence n in slot slots[n] (slots == NULL:
// slot n).  A slot outside [0, num_slots) is a padding entry: its output row
// is written as zeros and no state is touched.
struct DecodeArgs {
  const void *q, *k, *v;   // [N, Hqk, Dk], [N, Hqk, Dk], [N, Hv, Dv]
  const float *g, *beta;   // [N, Hv] (KDA g: [N, Hv, Dk]), [N, Hv]
  float *state;            // [num_slots, Hv, Dk, Dv], read and updated in place
  const int32_t *slots;    // [N] or NULL
  int N, Hqk, Hv, Dk, Dv, num_slots;
  float scale;
  int pre;                 // preprocessing flags (kPre*)
  void *o;                 // [N, Hv, Dv]
};

// Host-side launchers, one per kernel; each picks the template instance for
// (dtype, Dk, Dv, gate kind) and enqueues on `stream`.
hipError_t launch_chunk_index(const PrefillArgs &a, hipStream_t stream);
hipError_t launch_chunk_local(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
// ops #5 + #6 over whole chains (every sequence one segment)
hipError_t launch_state_prop(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
// launch_overlapped has instances for GDN in bf16 with Dk = Dv = 128 (KDA's
// chunk-local items are about twice as heavy and the overlapped launch measured
// slower for it: 185 against 116 us at 4096 tokens x 16 heads).
inline bool overlap_supported(bool bf16, bool kda, int Dk, int Dv) {
  return bf16 && !kda && Dk == 128 && Dv == 128;
}
// Zeroes the overlap queues and flags (and for a single sequence writes the
// device status word, which no chunk index kernel then writes).
hipError_t launch_overlap_setup(const PrefillArgs &a, hipStream_t stream);
// Chunk-local items and whole-chain walks in one launch (k1_chunk_local.hip).
hipError_t launch_overlapped(const PrefillArgs &a, hipStream_t stream);
// the bf16 whole-chain walk for batches with more walks than the device's
// compute units (a.cus; k2_walk.hip)
hipError_t launch_state_walk(const PrefillArgs &a, bool kda, int cus, hipStream_t stream);
// the bf16 segment maps on the staged walk (k2_walk.hip)
hipError_t launch_seg_maps(const PrefillArgs &a, bool kda, hipStream_t stream);
// segment-parallel path: segment maps, then ops #5 + #6 per segment
hipError_t launch_seg_transfer(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
hipError_t launch_seg_state(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
// one decode step (N x Hv x Dv/64 workgroups)
hipError_t launch_decode(const DecodeArgs &a, bool bf16, bool kda, hipStream_t stream);
// measured ceilings (k5_peaks.hip): a streaming copy of `bytes` (a multiple of
// 16) on 8 workgroups per CU, and `blocks` workgroups of four waves running
// `iters` rounds of 8 independent bf16 MFMAs each
hipError_t launch_copy(const void *src, void *dst, size_t bytes, int cus, hipStream_t stream);
hipError_t launch_mfma_loop(int blocks, int iters, float *sink, hipStream_t stream);

}  // namespace hagdn
