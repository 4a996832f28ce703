// k2_state_prop.hip -- the Reduce phase of chunkwise delta-rule prefill
// (paper Sec. 2.1, operator #5 H), the only step that is sequential over
// chunks, fused with the final Map (operator #6 O), for chains walked whole.
// One workgroup per (sequence, value head, 16-column tile of d_v); the tile's
// columns are dv_of(tile, 0..15) (device.h).  bf16 batches with more walks
// than CUs take the staged walk of k2_walk.hip, which shares a chunk's
// operands among several tiles of a head.  Chains long enough to pay for
// segment maps take the segment-parallel path of k3_segments.hip instead.
//
// Per chunk the chunk-local kernel has reduced operator #5 to an affine map of
// the state entering the chunk (S^T, d_k x d_v):
//     S^T_{c+1} = D S^T_c + NM S^T_c + B,     NM = -Kt W,  B = Kt U~,  D = Diag(e^gamma_last)
// so the critical path of one chunk step is a single d_k x d_k by d_k x 16
// product; nothing else waits on the state.
//
// Column split (paper Sec. 4, "Computation Splitting"): the columns of S^T
// (d_v) are independent, so a head splits into d_v/16 independent chains with
// no reduction between them.  Inside a chain, the DK/32 waves of the
// workgroup split the rows: wave w owns rows [32w, 32w+32) of the state tile,
// kept as two fp32 MFMA accumulator tiles for the whole sequence (the state
// never round-trips to HBM).  Per step each wave
//   1. rounds its rows to one B fragment (its 32-row k-block of S_c); with the
//      fragment layout of device.h the accumulator pair IS that fragment,
//      lane for lane,
//   2. stores it as the snapshot S_c for operator #6 and publishes it in LDS,
//   3. after one barrier, reads the other waves' fragments and computes its
//      rows of the next state: acc = D*S + B (fp32), acc += NM[rows][:] S_c.
// Chunk-first order (paper Sec. 5, "Cross-Chunk"): S_c is read by everything
// that needs it before its rows are overwritten -- including operator #6.
// After the exchange every wave holds all of S_c (this tile's 16 columns) as
// MFMA fragments, which are also the A operand of the output product
//     O^T = S_c Q'^T + O_loc^T        (operator #6, factors from the chunk-local kernel)
// so wave w emits its 16-token tile(s) of o in the same step, off the state's
// critical path.  The state is never written to memory between chunks.
//
// Latency: NM rows, the B tile and the decay do not depend on the state, so
// each wave keeps D chunks of them in flight in registers.  Loads are issued
// unconditionally (chunk index clamped) in a loop unrolled by D, so every
// path has the same number of memory operations in flight and each step waits
// only for its own chunk's operands.
//
// Workgroup -> (pair, tile) mapping is XCD-aware: consecutive workgroup ids
// are dealt round-robin to the 8 XCDs, so ids b, b+8, b+16, ... share an XCD;
// all d_v tiles of one (sequence, head) pair get ids in one such class and
// share that XCD's L2 for NM, which every tile of the pair reads.

#include "state_walk.h"

namespace hagdn {

template <typename T, int DK, int DV, bool KDA, bool SINGLE>
__global__ __launch_bounds__(64 * (DK / 32), sizeof(T) == 2 ? 2 : 1) void state_prop_kernel(PrefillArgs a) {
  constexpr int NT = DV / 16;  // d_v tiles per head
  single_status<SINGLE>(a);
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / NT) * kXcds + xcd;
  const int tile = slot % NT;
  if (pair >= a.N * a.Hv) return;  // uniform for the workgroup
  walk_tile<T, DK, DV, KDA, SINGLE, false>(a, pair, tile);
}

template <typename T, int DK, int DV, bool KDA>
static hipError_t launch_state_t(const PrefillArgs &a, hipStream_t stream) {
  const long pairs = (long)a.N * a.Hv;
  const long groups = (pairs + kXcds - 1) / kXcds;
  const long blocks = groups * kXcds * (DV / 16);
  if (a.single)
    hipLaunchKernelGGL((state_prop_kernel<T, DK, DV, KDA, true>), dim3((unsigned)blocks), dim3(64 * (DK / 32)), 0,
                       stream, a);
  else
    hipLaunchKernelGGL((state_prop_kernel<T, DK, DV, KDA, false>), dim3((unsigned)blocks), dim3(64 * (DK / 32)), 0,
                       stream, a);
  return hipGetLastError();
}

template <typename T, bool KDA>
static hipError_t dispatch_dims(const PrefillArgs &a, hipStream_t s) {
  if (a.Dk == 64 && a.Dv == 64) return launch_state_t<T, 64, 64, KDA>(a, s);
  if (a.Dk == 64 && a.Dv == 128) return launch_state_t<T, 64, 128, KDA>(a, s);
  if (a.Dk == 128 && a.Dv == 64) return launch_state_t<T, 128, 64, KDA>(a, s);
  return launch_state_t<T, 128, 128, KDA>(a, s);
}

hipError_t launch_state_prop(const PrefillArgs &a, bool bf16, bool kda, hipStream_t s) {
  if (bf16) {
    // more walks than CUs: the staged walk, several tiles per workgroup
    const long walks = ((long)a.N * a.Hv + kXcds - 1) / kXcds * kXcds * (a.Dv / 16);
    if (walks > a.cus) return launch_state_walk(a, kda, a.cus, s);
    return kda ? dispatch_dims<bf16_t, true>(a, s) : dispatch_dims<bf16_t, false>(a, s);
  }
  return kda ? dispatch_dims<float, true>(a, s) : dispatch_dims<float, false>(a, s);
}

}  // namespace hagdn
