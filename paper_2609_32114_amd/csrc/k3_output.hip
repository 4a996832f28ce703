// k3_output.hip -- the final Map phase of chunkwise delta-rule prefill
// (paper Sec. 2.1, operator #6 O), one workgroup per (chunk, value head),
// fully parallel.  Operator #6 needs only the state S_c entering the chunk
// and chunk-local factors (paper Sec. 5, "Cross-Chunk"); with the factors of
// the chunk-local kernel it is one product:
//
//   O = scale * (Q' S^T_c + O_loc),   Q' = Q * e^gamma - P W,  O_loc = P U~
//
// computed transposed, O^T = S_c Q'^T + O_loc^T, so that each lane's
// accumulator holds 4 consecutive d_v values of one token (an 8-byte bf16
// store into o[token][head][d_v]).  The snapshot S_c, Q' and O_loc arrive in
// fragment order (prefill.h): every operand load is one contiguous 1 KiB run
// per wave, and the S_c and Q' fragments pair directly.  Wave w owns d_v rows
// [w*DV/4, (w+1)*DV/4) for all 64 tokens.
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kOutThreads = 256;

template <typename T, int DK, int DV>
__global__ __launch_bounds__(kOutThreads) void output_kernel(PrefillArgs a) {
  constexpr int MPW = DV / 16 / 4;  // 16-row d_v tiles per wave
  const int c = blockIdx.x, h = blockIdx.y;
  const int4 ci = a.chunk_info[c];
  const int len = ci.z;
  if (len <= 0) return;
  const int start = ci.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const size_t blk = (size_t)c * a.Hv + h;
  const T *hs = static_cast<const T *>(a.Hs) + blk * ((size_t)DV * DK);
  const T *qp = static_cast<const T *>(a.Qp) + blk * ((size_t)kChunk * DK);
  const T *ol = static_cast<const T *>(a.Ol) + blk * ((size_t)kChunk * DV);
  T *o = static_cast<T *>(a.o);

#pragma unroll
  for (int mi = 0; mi < MPW; ++mi) {
    const int m = wave * MPW + mi;      // d_v tile
    Frag<T> sa[DK / 32];  // snapshot blocks (d_v tile m, kb), fragment order
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) sa[kb] = load_frag_at(hs + ((size_t)(m * (DK / 32) + kb) * 64 + lane) * 8);
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) {    // token tile
      const int r = 16 * nt + col;      // token this lane's accumulator column holds
      f32x4 acc = load4(ol + ((size_t)(nt * (DV / 16) + m) * 64 + lane) * 4);
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb)
        acc = mma(acc, sa[kb], load_frag_at(qp + ((size_t)(nt * (DK / 32) + kb) * 64 + lane) * 8));
      if (r < len) store4(o + ((size_t)(start + r) * a.Hv + h) * DV + 16 * m + 4 * grp, acc * a.scale);
    }
  }
}

template <typename T, int DK, int DV>
static hipError_t launch_output_t(const PrefillArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL((output_kernel<T, DK, DV>), dim3(a.max_chunks, a.Hv), dim3(kOutThreads), 0,
                     stream, a);
  return hipGetLastError();
}

template <typename T>
static hipError_t dispatch_dims(const PrefillArgs &a, hipStream_t s) {
  if (a.Dk == 64 && a.Dv == 64) return launch_output_t<T, 64, 64>(a, s);
  if (a.Dk == 64 && a.Dv == 128) return launch_output_t<T, 64, 128>(a, s);
  if (a.Dk == 128 && a.Dv == 64) return launch_output_t<T, 128, 64>(a, s);
  return launch_output_t<T, 128, 128>(a, s);
}

hipError_t launch_output(const PrefillArgs &a, bool bf16, hipStream_t s) {
  if (a.max_chunks == 0) return hipSuccess;
  return bf16 ? dispatch_dims<bf16_t>(a, s) : dispatch_dims<float>(a, s);
}

}  // namespace hagdn
