// k4_decode.hip -- one decode step of the delta rule: a single new token for
// each of N sequences, advanced by the token-by-token recurrence that serves
// decoding (paper Sec. 2.1; Sec. 7.3 leaves decode to the serving backend, so
// this is the step after the prefill hot path, starting from its final state).
//
// Per (sequence n, value head h), with H = S^T the d_k x d_v state of slot
// slots[n] and a = e^g (a d_k-vector for KDA, acting on the rows of H):
//   H' = Diag(a) H;   p = H'^T k;   u = b (v - p);   H'' = H' + k u^T;
//   o  = scale H''^T q,   H <- H''   (in place)
// Every state column is independent: column c needs only column c of H and
// the two reductions over the d_k rows (p_c, then o_c).  One workgroup owns
// 64 columns of one (sequence, head): thread (row group rg, column group cg)
// holds rows rg + 16 i of columns 4cg .. 4cg+3 as float4s, so each wave
// instruction moves four full 256-byte row segments.  The step is bound by
// HBM: 8 d_k d_v bytes of state per head against ~4 d_k d_v flops.  The state
// is streamed with nontemporal loads and stores: a decode batch's states are
// touched once per step, and keeping them out of the caches measured faster
// once the pool outgrows the Infinity Cache (0.96x the time at 256 MiB).
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kDecThreads = 256;
constexpr int kDecCols = 64;  // state columns per workgroup

template <typename T, int DK, int DV, bool KDA>
__global__ __launch_bounds__(kDecThreads) void decode_kernel(DecodeArgs a) {
  using E = Elt<T>;
  constexpr int TILES = DV / kDecCols;
  constexpr int CG = kDecCols / 4;        // column groups of 4
  constexpr int RG = kDecThreads / CG;    // row groups
  constexpr int RPT = DK / RG;            // rows per thread
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int cg = tid % CG, rg = tid / CG;
  const int tile = blockIdx.x % TILES;
  const int nh = blockIdx.x / TILES;
  const int n = nh / a.Hv, h = nh % a.Hv;
  const int hk = h / (a.Hv / a.Hqk);
  const int c0 = tile * kDecCols + 4 * cg;
  __shared__ f32x4 sP[4][CG], sO[4][CG];

  T *o = static_cast<T *>(a.o) + ((size_t)n * a.Hv + h) * DV + c0;
  const int slot = a.slots ? a.slots[n] : n;
  if (slot < 0 || slot >= a.num_slots) {  // padding entry: uniform over the workgroup
    if (rg == 0) store4(o, zero4());
    return;
  }
  float *S = a.state + ((size_t)slot * a.Hv + h) * DK * DV + c0;
  f32x4 H[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    H[i] = __builtin_nontemporal_load(reinterpret_cast<const f32x4 *>(S + (size_t)(rg + RG * i) * DV));

  const T *qh = static_cast<const T *>(a.q) + ((size_t)n * a.Hqk + hk) * DK;
  const T *kh = static_cast<const T *>(a.k) + ((size_t)n * a.Hqk + hk) * DK;
  float kr[RPT], qr[RPT], ar[RPT];
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    kr[i] = E::to_f32(kh[rg + RG * i]);
    qr[i] = E::to_f32(qh[rg + RG * i]);
  }
  const size_t nhi = (size_t)n * a.Hv + h;
  float b = a.beta[nhi];
  const f32x4 vv = load4(static_cast<const T *>(a.v) + nhi * DV + c0);
  if constexpr (KDA) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) ar[i] = a.g[nhi * DK + rg + RG * i];
  } else {
    const float gv = a.g[nhi];
#pragma unroll
    for (int i = 0; i < RPT; ++i) ar[i] = gv;
  }

  if (a.pre & kPreQkNorm) {  // each wave forms both norms itself
    float sq = 0.f, sk = 0.f;
#pragma unroll
    for (int d = lane; d < DK; d += 64) {
      const float x = E::to_f32(qh[d]), y = E::to_f32(kh[d]);
      sq += x * x;
      sk += y * y;
    }
    const float iq = inv_l2(wave_sum(sq)), ik = inv_l2(wave_sum(sk));
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      qr[i] *= iq;
      kr[i] *= ik;
    }
  }
  if (a.pre & kPreGateSoftplus) {
#pragma unroll
    for (int i = 0; i < RPT; ++i) ar[i] = neg_softplus(ar[i]);
  }
  if (a.pre & kPreBetaSigmoid) b = sigmoid(b);
#pragma unroll
  for (int i = 0; i < RPT; ++i) ar[i] = expf(ar[i]);

  // p = (Diag(a) H)^T k over this thread's rows, then over the wave's row
  // groups (lanes CG apart), then over the four waves
  f32x4 p = zero4();
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    H[i] *= ar[i];
    p += H[i] * kr[i];
  }
#pragma unroll
  for (int off = CG; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 4; ++e) p[e] += __shfl_xor(p[e], off);
  if (lane < CG) sP[wave][lane] = p;
  __syncthreads();
  const f32x4 pt = sP[0][cg] + sP[1][cg] + sP[2][cg] + sP[3][cg];
  const f32x4 u = b * (vv - pt);

  f32x4 ov = zero4();
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    H[i] += kr[i] * u;
    ov += H[i] * qr[i];
    __builtin_nontemporal_store(H[i], reinterpret_cast<f32x4 *>(S + (size_t)(rg + RG * i) * DV));
  }
#pragma unroll
  for (int off = CG; off < 64; off <<= 1)
#pragma unroll
    for (int e = 0; e < 4; ++e) ov[e] += __shfl_xor(ov[e], off);
  if (lane < CG) sO[wave][lane] = ov;
  __syncthreads();
  if (tid < CG) store4(o, a.scale * (sO[0][cg] + sO[1][cg] + sO[2][cg] + sO[3][cg]));
}

template <typename T, bool KDA>
static hipError_t launch_decode_t(const DecodeArgs &a, hipStream_t s) {
  const unsigned grid = (unsigned)((size_t)a.N * a.Hv * (a.Dv / kDecCols));
#define HAGDN_DEC(DK_, DV_)                                                                          \
  hipLaunchKernelGGL((decode_kernel<T, DK_, DV_, KDA>), dim3(grid), dim3(kDecThreads), 0, s, a); \
  return hipGetLastError()
  if (a.Dk == 64 && a.Dv == 64) { HAGDN_DEC(64, 64); }
  if (a.Dk == 64 && a.Dv == 128) { HAGDN_DEC(64, 128); }
  if (a.Dk == 128 && a.Dv == 64) { HAGDN_DEC(128, 64); }
  HAGDN_DEC(128, 128);
#undef HAGDN_DEC
}

hipError_t launch_decode(const DecodeArgs &a, bool bf16, bool kda, hipStream_t s) {
  if (a.N == 0) return hipSuccess;
  if (bf16) return kda ? launch_decode_t<bf16_t, true>(a, s) : launch_decode_t<bf16_t, false>(a, s);
  return kda ? launch_decode_t<float, true>(a, s) : launch_decode_t<float, false>(a, s);
}

}  // namespace hagdn
