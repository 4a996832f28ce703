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
// `blk = chunk * Hv + h` each region holds one fixed-size block:
//   W   [64][Dk]    -W, W = T Diag(b) (K * e^gamma)   (op #4; Sec. 5 "W = A^-1 K")
//   Ut  [Dv][64]    U~^T, U~ = T Diag(b) V            (op #4)
//   Kt  [Dk][64]    (K * e^(gamma_last - gamma))^T    (keys as op #5-update uses them)
//   Qt  [64][Dk]    Q * e^gamma                       (queries as op #6 uses them)
//   P   [64][64]    P[r][s] = <q_r, e^(gamma_r-gamma_s) k_s>, s <= r, else 0
//   dec [Dk]        e^gamma_last (GDN: element 0 only)
//   U   [Dv][64]    U^T, U = U~ - W S_c^T  (the "v_c" of op #5-read, Sec. 5)
//   Hs  [Dv][Dk]    S_c, the state entering the chunk (snapshot for op #6)
// Element type of every block is the I/O dtype (bf16 or fp32).  Inside each
// 32-block along the contracted index, W (d_k), Kt (tokens), Qt (d_k), P
// (tokens), U (tokens) and Hs (d_k) are kmap-permuted (device.h): W and Kt
// pair with accumulator-derived fragments in the state kernel, U and Hs are
// written as those fragments, Qt and P pair with them in the output kernel.
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
  void *W, *Ut, *Kt, *Qt, *P, *U, *Hs;
  float *dec;
};

// Host-side launchers, one per kernel; each picks the template instance for
// (dtype, Dk, Dv, gate kind) and enqueues on `stream`.
hipError_t launch_chunk_index(const PrefillArgs &a, hipStream_t stream);
hipError_t launch_chunk_local(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
hipError_t launch_state_prop(const PrefillArgs &a, bool bf16, bool kda, hipStream_t stream);
hipError_t launch_output(const PrefillArgs &a, bool bf16, hipStream_t stream);

}  // namespace hagdn
