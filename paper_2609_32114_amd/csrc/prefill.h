// prefill.h -- internal interface between the host launcher (api.cpp) and the
// HIP kernels.  Not part of the public ABI (that is include/hagdn.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace hagdn {

constexpr int kChunk = 64;  // chunk length C (paper Sec. 7.1 uses C = 64)

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
// NM, Bc, Qp and Ol are stored in fragment order (device.h): one 16-lane
// by 32 (operands) or 16x16 (accumulators) block after another, 64 lanes x 8
// (operand) or x 4 (accumulator) elements each, so every producer and consumer
// moves whole blocks with contiguous 16- or 8-byte lane accesses:
//   NM  operand blocks (row tile t of d_k out, k-block kb of d_k in), t-major;
//       slot j of lane (col, grp) = NM[16t + col][32kb + kmap(grp, j)]
//   Bc  accumulator blocks (d_v tile n, d_k tile m), n-major;
//       element e of lane (col, grp) = B[16m + 4grp + e][16n + col]
//   Qp  operand blocks (token tile nt, k-block kb of d_k), nt-major;
//       slot j of lane (col, grp) = Q'[16nt + col][32kb + kmap(grp, j)]
//   Ol  accumulator blocks (token tile nt, d_v tile m), nt-major;
//       element e of lane (col, grp) = O_loc[16nt + col][16m + 4grp + e]
// Element type of every block is the I/O dtype (bf16 or fp32), dec is fp32.
struct PrefillArgs {
  const void *q, *k, *v;
  const float *g, *beta, *s0;
  const int32_t *cu_seqlens;
  int N, T, Hqk, Hv, Dk, Dv;
  int max_chunks;  // upper bound on chunks: T / 64 + N
  float scale;
  void *o;
  float *s_final;
  // workspace
  int *status;         // [1] device status word (hagdn_device_code)
  int4 *seq_info;      // [N]  {first chunk, number of chunks, start token, length}
  int4 *chunk_info;    // [max_chunks] {sequence, start token, length, 0}; length 0 = unused
  void *NM, *Bc, *Qp, *Ol;
  float *dec;
};

// Host-side launchers, one per kernel; each picks the template instance for
// (dtype, Dk, Dv, gate kind) and enqueues on `stream`.
hipError_t launch_chunk_index(const PrefillArgs &a, hipStream_t stream);
hipError_t launch_chunk_local(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
hipError_t launch_state_prop(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);  // ops #5 + #6

}  // namespace hagdn
