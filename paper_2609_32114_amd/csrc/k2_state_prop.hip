// k2_state_prop.hip -- the Reduce phase of chunkwise delta-rule prefill
// (paper Sec. 2.1, operator #5 H): the only step that is sequential over
// chunks.  One wave per (sequence, value head, 16-column tile of d_v).
//
// Column split (paper Sec. 4, "Computation Splitting"): the columns of the
// state S^T (d_v) are independent -- every product below contracts over d_k
// or over tokens, never over d_v -- so a head splits into d_v/16 independent
// chains with no cross-wave reduction.  The state tile (d_k x 16, fp32) lives
// in MFMA accumulators for the whole sequence and never round-trips to HBM.
//
// Chunk-first order (paper Sec. 5, "Cross-Chunk"): per chunk the state is
// read for everything that needs S_c before it is updated in place:
//   5-read   snapshot S_c (for operator #6), U = U~ - W S_c^T  ("v_c")
//   5-update S^T <- Diag(e^gamma_last) S^T + Kt U
// With the fragment layout of device.h, the accumulator tiles of S^T are
// directly the B operand of W S_c^T and the accumulator tiles of U are
// directly the B operand of Kt U: no LDS round trip, no lane shuffles.
//
// Workgroup -> (pair, tile) mapping is XCD-aware: consecutive workgroup ids
// are dealt round-robin to the 8 XCDs, so ids b, b+8, b+16, ... share an XCD;
// all d_v tiles of one (sequence, head) pair get ids in one such class and
// share that XCD's L2 for W and Kt, which every tile of the pair reads.
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kXcds = 8;

template <typename T, int DK, int DV, bool KDA>
__global__ __launch_bounds__(64) void state_prop_kernel(PrefillArgs a) {
  constexpr int NT = DV / 16;   // d_v tiles per head
  constexpr int KT = DK / 16;   // accumulator tiles of the state (d_k rows)
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / NT) * kXcds + xcd;
  const int tile = slot % NT;
  if (pair >= a.N * a.Hv) return;
  const int n = pair / a.Hv, h = pair % a.Hv;
  const int lane = threadIdx.x, col = lane & 15, grp = lane >> 4;
  const int dv = tile * 16 + col;  // state column this lane holds
  const int4 si = a.seq_info[n];   // {first chunk, chunks, start, length}

  // state tile: H[t][e] = S^T[16t + 4grp + e][dv]
  f32x4 H[KT];
  const size_t sbase = ((size_t)n * a.Hv + h) * DK * DV;
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      H[t][e] = a.s0 ? a.s0[sbase + (size_t)(16 * t + 4 * grp + e) * DV + dv] : 0.f;

  const T *Wg = static_cast<const T *>(a.W);
  const T *Utg = static_cast<const T *>(a.Ut);
  const T *Ktg = static_cast<const T *>(a.Kt);
  T *Ug = static_cast<T *>(a.U);
  T *Hsg = static_cast<T *>(a.Hs);

  for (int c = 0; c < si.y; ++c) {
    const size_t blk = (size_t)(si.x + c) * a.Hv + h;
    // 5-read: snapshot S_c (stored [d_v][d_k], what operator #6 reads)
    T *hs = Hsg + blk * ((size_t)DV * DK) + (size_t)dv * DK;
#pragma unroll
    for (int t = 0; t < KT; ++t) store4(hs + 16 * t + 4 * grp, H[t]);

    // U = U~ - W S_c^T   (rows = tokens, columns = this tile's d_v)
    Frag<T> hb[DK / 32];
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) hb[kb] = frag_from_acc<T>(H[2 * kb], H[2 * kb + 1], -1.f);
    const T *ut = Utg + blk * ((size_t)DV * kChunk) + (size_t)dv * kChunk;
    const T *w = Wg + blk * ((size_t)kChunk * DK);
    f32x4 U[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      U[m] = load4(ut + 16 * m + 4 * grp);
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb)
        U[m] = mma(U[m], load_frag(w + (size_t)(16 * m + col) * DK + kb * 32, grp), hb[kb]);
    }
    // U in the operand precision: stored for operator #6 and used below
    T *uo = Ug + blk * ((size_t)DV * kChunk) + (size_t)dv * kChunk;
#pragma unroll
    for (int m = 0; m < 4; ++m) store4(uo + 16 * m + 4 * grp, U[m]);
    Frag<T> ub[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) ub[kb] = frag_from_acc<T>(U[2 * kb], U[2 * kb + 1], 1.f);

    // 5-update: S^T <- Diag(e^gamma_last) S^T + Kt U
    const float *dec = a.dec + blk * DK;
    if constexpr (KDA) {
#pragma unroll
      for (int t = 0; t < KT; ++t) H[t] *= load4(dec + 16 * t + 4 * grp);
    } else {
      const float d0 = dec[0];
#pragma unroll
      for (int t = 0; t < KT; ++t) H[t] *= d0;
    }
    const T *kt = Ktg + blk * ((size_t)DK * kChunk);
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        H[t] = mma(H[t], load_frag(kt + (size_t)(16 * t + col) * kChunk + kb * 32, grp), ub[kb]);
  }

  if (a.s_final) {
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        a.s_final[sbase + (size_t)(16 * t + 4 * grp + e) * DV + dv] = H[t][e];
  }
}

template <typename T, int DK, int DV, bool KDA>
static hipError_t launch_state_t(const PrefillArgs &a, hipStream_t stream) {
  const long pairs = (long)a.N * a.Hv;
  const long groups = (pairs + kXcds - 1) / kXcds;
  const long blocks = groups * kXcds * (DV / 16);
  hipLaunchKernelGGL((state_prop_kernel<T, DK, DV, KDA>), dim3((unsigned)blocks), dim3(64), 0,
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
  if (bf16) return kda ? dispatch_dims<bf16_t, true>(a, s) : dispatch_dims<bf16_t, false>(a, s);
  return kda ? dispatch_dims<float, true>(a, s) : dispatch_dims<float, false>(a, s);
}

}  // namespace hagdn
