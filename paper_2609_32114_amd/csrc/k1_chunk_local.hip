// k1_chunk_local.hip -- the first Map phase of chunkwise delta-rule prefill
// (paper Sec. 2.1: operators #1 Gate, #2 KKT, #3 Solve, #4 W/U), one
// workgroup per (chunk, value head), fully parallel over both.
//
// For a chunk of n <= 64 tokens (rows >= n are zero-padded, which makes them
// contribute nothing downstream), with gamma the inclusive cumulative
// log-gate inside the chunk (a d_k-vector per token for KDA):
//   #1  gamma_r = sum_{s<=r} g_s
//   #2  A[r][s] = b_r <k_r, e^(gamma_r - gamma_s) k_s>           (s < r)
//       P[r][s] =     <q_r, e^(gamma_r - gamma_s) k_s>           (s <= r)
//   #3  T = (I + A)^-1                       (unit lower triangular, fp32)
//   #4  W  = T Diag(b) (K * e^gamma)         U~ = T Diag(b) V
// plus the operands the sequential kernel and the output kernel consume:
//   Kt = (K * e^(gamma_last - gamma))^T,  Qt = Q * e^gamma,  dec = e^gamma_last.
// W and Kt are the A operands of the state kernel's chained products and are
// stored kmap-permuted inside each 32-block (see device.h), W negated; Qt and P
// are the partners of the state kernel's fragment-order outputs (snapshot,
// corrected values) in the output kernel and are kmap-permuted along d_k and
// along tokens respectively.  Ut is stored in logical order.
// P is the decay-masked Q K^T of Sec. 5's GEMM group (KK^T and QK^T share K
// and are computed together); the solve never has to wait on a GEMM input.
//
// GDN's decay is a scalar per token, so K K^T and Q K^T are plain MFMA
// products and the decay is applied in the epilogue.  KDA's per-channel decay
// sits inside the contraction: off-diagonal 16x16 blocks factor it around the
// first token rho of the row block, <k_r e^(gamma_r - gamma_rho),
// k_s e^(gamma_rho - gamma_s)>, both factors <= 1; diagonal blocks are summed
// elementwise in fp32 (their exponents are clamped at 0 before masking).
//
// Wave roles (4 waves): wave i computes row block i of A and P; wave 0 then
// solves T by forward substitution (lane j owns column j) while waves 1-3
// write Kt, Qt and dec; finally wave i computes token block i of W and U~.
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kLocalThreads = 256;

template <typename T, int DK, int DV, bool KDA>
struct LocalLayout {
  static constexpr int PAD = 16 / (int)sizeof(T);
  static constexpr int LDK = DK + PAD;       // sK   [64][LDK]   keys, token rows
  static constexpr int LDT = kChunk + PAD;   // sKt  [DK][LDT]   keys, channel rows
                                             // sVt  [DV][LDT]   values, channel rows
  static constexpr int LDA = kChunk + 4;     // sA   [64][LDA]   A, then T (fp32)
  static constexpr int LDG = KDA ? DK + 1 : 1;  // sGam [64][LDG] (GDN: [64])
  static constexpr size_t off_K = 0;
  static constexpr size_t off_Kt = off_K + sizeof(T) * kChunk * LDK;
  static constexpr size_t off_Vt = off_Kt + sizeof(T) * DK * LDT;
  static constexpr size_t off_A = off_Vt + sizeof(T) * DV * LDT;
  static constexpr size_t off_beta = off_A + sizeof(float) * kChunk * LDA;
  static constexpr size_t off_gam = off_beta + sizeof(float) * kChunk;
  static constexpr size_t bytes = off_gam + sizeof(float) * kChunk * LDG;
};

template <typename T, int DK, int DV, bool KDA>
__global__ __launch_bounds__(kLocalThreads) void chunk_local_kernel(PrefillArgs a) {
  using L = LocalLayout<T, DK, DV, KDA>;
  using E = Elt<T>;
  constexpr int V = 16 / (int)sizeof(T);  // elements per 16-byte vector
  const int c = blockIdx.x, h = blockIdx.y;
  const int4 ci = a.chunk_info[c];
  const int len = ci.z;
  if (len <= 0) return;
  const int start = ci.y;
  const int hk = h / (a.Hv / a.Hqk);
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const size_t blk = (size_t)c * a.Hv + h;

  extern __shared__ __align__(16) unsigned char smem[];
  T *sK = reinterpret_cast<T *>(smem + L::off_K);
  T *sKt = reinterpret_cast<T *>(smem + L::off_Kt);
  T *sVt = reinterpret_cast<T *>(smem + L::off_Vt);
  float *sA = reinterpret_cast<float *>(smem + L::off_A);
  float *sBeta = reinterpret_cast<float *>(smem + L::off_beta);
  float *sGam = reinterpret_cast<float *>(smem + L::off_gam);

  const size_t qk_row = (size_t)a.Hqk * DK;  // token stride of q and k
  const size_t v_row = (size_t)a.Hv * DV;
  const T *kbase = static_cast<const T *>(a.k) + (size_t)start * qk_row + (size_t)hk * DK;
  const T *qbase = static_cast<const T *>(a.q) + (size_t)start * qk_row + (size_t)hk * DK;
  const T *vbase = static_cast<const T *>(a.v) + (size_t)start * v_row + (size_t)h * DV;

  // ---- stage K (token rows and channel rows) and V (channel rows)
  for (int idx = tid; idx < kChunk * DK / V; idx += kLocalThreads) {
    const int r = idx / (DK / V), cv = (idx % (DK / V)) * V;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (r < len) u = *reinterpret_cast<const uint4 *>(kbase + (size_t)r * qk_row + cv);
    *reinterpret_cast<uint4 *>(sK + r * L::LDK + cv) = u;
#pragma unroll
    for (int j = 0; j < V; ++j) sKt[(cv + j) * L::LDT + r] = Vec16<T>::raw(u, j);
  }
  for (int idx = tid; idx < kChunk * DV / V; idx += kLocalThreads) {
    const int r = idx / (DV / V), cv = (idx % (DV / V)) * V;
    uint4 u = make_uint4(0, 0, 0, 0);
    if (r < len) u = *reinterpret_cast<const uint4 *>(vbase + (size_t)r * v_row + cv);
#pragma unroll
    for (int j = 0; j < V; ++j) sVt[(cv + j) * L::LDT + r] = Vec16<T>::raw(u, j);
  }

  // ---- op #1: beta and gamma (padded tokens: g = 0, b = 0)
  if (tid < kChunk) sBeta[tid] = tid < len ? a.beta[(size_t)(start + tid) * a.Hv + h] : 0.f;
  if constexpr (!KDA) {
    if (wave == 0) {
      float x = lane < len ? a.g[(size_t)(start + lane) * a.Hv + h] : 0.f;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const float y = __shfl_up(x, off);
        if (lane >= off) x += y;
      }
      sGam[lane] = x;
    }
  } else {
    const float *gb = a.g + ((size_t)start * a.Hv + h) * DK;
    const size_t g_row = (size_t)a.Hv * DK;
    for (int d = tid; d < DK; d += kLocalThreads) {
      float acc = 0.f;
#pragma unroll 8
      for (int r = 0; r < kChunk; ++r) {
        if (r < len) acc += gb[(size_t)r * g_row + d];
        sGam[r * L::LDG + d] = acc;
      }
    }
  }
  __syncthreads();

  // ---- op #2: A (into LDS) and P (to the workspace); wave i = row block i
  T *Pout = static_cast<T *>(a.P) + blk * (kChunk * kChunk);
  {
    const int i = wave, r0 = 16 * i, ra = r0 + col;
    const T *qrow = qbase + (size_t)ra * qk_row;
    if constexpr (!KDA) {
      Frag<T> ka[DK / 32], qa[DK / 32];
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb) {
        ka[kb] = load_frag(sK + ra * L::LDK + kb * 32, grp);
        qa[kb] = ra < len ? load_frag(qrow + kb * 32, grp) : zero_frag<T>();
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        f32x4 accA = zero4(), accP = zero4();
        if (j <= i) {
#pragma unroll
          for (int kb = 0; kb < DK / 32; ++kb) {
            const Frag<T> kf = load_frag(sK + (16 * j + col) * L::LDK + kb * 32, grp);
            accA = mma(accA, ka[kb], kf);
            accP = mma(accP, qa[kb], kf);
          }
        }
        const int s = 16 * j + col;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + 4 * grp + e;
          float vA = 0.f, vP = 0.f;
          if (s <= r) {
            const float dec = __expf(sGam[r] - sGam[s]);
            vP = accP[e] * dec;
            if (s < r) vA = sBeta[r] * accA[e] * dec;
          }
          sA[r * L::LDA + s] = vA;
          Pout[r * kChunk + (s & ~31) + kmap_pos(s & 31)] = E::from_f32(vP);
        }
      }
    } else {
      const int rho = r0;  // reference token of this row block
      Frag<T> ka[DK / 32], qa[DK / 32];
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb) {
        float xk[8], xq[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int d = kb * 32 + kc(grp, j);
          const float ex = __expf(sGam[ra * L::LDG + d] - sGam[rho * L::LDG + d]);
          xk[j] = E::to_f32(sK[ra * L::LDK + d]) * ex;
          xq[j] = ra < len ? E::to_f32(qrow[d]) * ex : 0.f;
        }
        ka[kb] = make_frag<T>(xk);
        qa[kb] = make_frag<T>(xq);
      }
      for (int j = 0; j < i; ++j) {  // off-diagonal blocks: factored decay
        f32x4 accA = zero4(), accP = zero4();
        const int sb = 16 * j + col;
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb) {
          float xb[8];
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const int d = kb * 32 + kc(grp, jj);
            xb[jj] = E::to_f32(sK[sb * L::LDK + d]) *
                     __expf(sGam[rho * L::LDG + d] - sGam[sb * L::LDG + d]);
          }
          const Frag<T> kf = make_frag<T>(xb);
          accA = mma(accA, ka[kb], kf);
          accP = mma(accP, qa[kb], kf);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + 4 * grp + e;
          sA[r * L::LDA + sb] = sBeta[r] * accA[e];
          Pout[r * kChunk + (sb & ~31) + kmap_pos(sb & 31)] = E::from_f32(accP[e]);
        }
      }
      {  // diagonal block: elementwise fp32
        const int s = r0 + col;
        float accA[4] = {0.f, 0.f, 0.f, 0.f}, accP[4] = {0.f, 0.f, 0.f, 0.f};
        for (int d = 0; d < DK; ++d) {
          const float ks = E::to_f32(sK[s * L::LDK + d]);
          const float gs = sGam[s * L::LDG + d];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = r0 + 4 * grp + e;
            const float ex = __expf(fminf(sGam[r * L::LDG + d] - gs, 0.f));
            const float kr = E::to_f32(sK[r * L::LDK + d]);
            const float qr = r < len ? E::to_f32(qbase[(size_t)r * qk_row + d]) : 0.f;
            accA[e] += kr * ks * ex;
            accP[e] += qr * ks * ex;
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + 4 * grp + e;
          sA[r * L::LDA + s] = s < r ? sBeta[r] * accA[e] : 0.f;
          Pout[r * kChunk + (s & ~31) + kmap_pos(s & 31)] = E::from_f32(s <= r ? accP[e] : 0.f);
        }
      }
      for (int j = i + 1; j < 4; ++j) {  // above the diagonal: zero
        const int s = 16 * j + col;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + 4 * grp + e;
          sA[r * L::LDA + s] = 0.f;
          Pout[r * kChunk + (s & ~31) + kmap_pos(s & 31)] = E::from_f32(0.f);
        }
      }
    }
  }
  __syncthreads();

  if (wave == 0) {
    // ---- op #3: T = (I + A)^-1.  Lane j solves column j:
    //      x_r = delta_rj - sum_{s<r} A[r][s] x_s   (rows r < j give x_r = 0)
    float x[kChunk];
#pragma unroll
    for (int r = 0; r < kChunk; ++r) {
      const float *Ar = sA + r * L::LDA;
      float p0 = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll
      for (int s = 0; s + 3 < r; s += 4) {
        const f32x4 av = *reinterpret_cast<const f32x4 *>(Ar + s);
        p0 += av[0] * x[s];
        p1 += av[1] * x[s + 1];
        p2 += av[2] * x[s + 2];
        p3 += av[3] * x[s + 3];
      }
#pragma unroll
      for (int s = r & ~3; s < r; ++s) p0 += Ar[s] * x[s];
      x[r] = (r == lane ? 1.f : 0.f) - ((p0 + p1) + (p2 + p3));
    }
#pragma unroll
    for (int r = 0; r < kChunk; ++r) sA[r * L::LDA + lane] = x[r];
  } else {
    // ---- operands for the sequential and output kernels (threads 64..255)
    const int t2 = tid - 64;
    T *kt_out = static_cast<T *>(a.Kt) + blk * ((size_t)DK * kChunk);
    for (int idx = t2; idx < DK * kChunk / V; idx += kLocalThreads - 64) {
      // output positions p0..p0+V-1 of row d; position p holds logical token
      // (p & ~31) + kmap((p & 31) >> 3, p & 7) -- the kmap-permuted layout the
      // state kernel pairs with its accumulator-derived U fragments
      const int d = idx / (kChunk / V), p0 = (idx % (kChunk / V)) * V;
      float outv[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int p = p0 + j;
        const int s = (p & ~31) + kmap((p & 31) >> 3, p & 7);
        const float ex = KDA ? __expf(sGam[(kChunk - 1) * L::LDG + d] - sGam[s * L::LDG + d])
                             : __expf(sGam[kChunk - 1] - sGam[s]);
        outv[j] = E::to_f32(sKt[d * L::LDT + s]) * ex;
      }
      *reinterpret_cast<uint4 *>(kt_out + (size_t)d * kChunk + p0) = Vec16<T>::pack(outv);
    }
    // Qt = Q * e^gamma, kmap-permuted along d_k: item (r, kb, g) writes the 8
    // elements at positions kb*32 + 8g + j, i.e. logical d = kb*32 + kmap(g, j),
    // read as two runs of 4 from q
    T *qt_out = static_cast<T *>(a.Qt) + blk * ((size_t)kChunk * DK);
    for (int idx = t2; idx < kChunk * DK / 8; idx += kLocalThreads - 64) {
      const int r = idx / (DK / 8), kb = (idx % (DK / 8)) >> 2, g = idx & 3;
      const int d0 = kb * 32 + 4 * g, d1 = kb * 32 + 16 + 4 * g;
      f32x4 x0 = zero4(), x1 = zero4();
      if (r < len) {
        x0 = load4(qbase + (size_t)r * qk_row + d0);
        x1 = load4(qbase + (size_t)r * qk_row + d1);
      }
      float outv[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        outv[j] = x0[j] * (KDA ? __expf(sGam[r * L::LDG + d0 + j]) : __expf(sGam[r]));
        outv[4 + j] = x1[j] * (KDA ? __expf(sGam[r * L::LDG + d1 + j]) : __expf(sGam[r]));
      }
      T *dst = qt_out + (size_t)r * DK + kb * 32 + 8 * g;
      if constexpr (sizeof(T) == 2) {
        *reinterpret_cast<uint4 *>(dst) = Vec16<T>::pack(outv);
      } else {
        const float a0[4] = {outv[0], outv[1], outv[2], outv[3]}, a1[4] = {outv[4], outv[5], outv[6], outv[7]};
        *reinterpret_cast<uint4 *>(dst) = Vec16<T>::pack(a0);
        *reinterpret_cast<uint4 *>(dst + 4) = Vec16<T>::pack(a1);
      }
    }
    float *dec_out = a.dec + blk * DK;
    if constexpr (KDA) {
      for (int d = t2; d < DK; d += kLocalThreads - 64)
        dec_out[d] = __expf(sGam[(kChunk - 1) * L::LDG + d]);
    } else {
      if (t2 == 0) dec_out[0] = __expf(sGam[kChunk - 1]);
    }
  }
  __syncthreads();

  // ---- op #4: wave i = token block i.  T' = T Diag(b) (GDN: also e^gamma_s)
  {
    const int i = wave, r = 16 * i + col;
    Frag<T> tu[2], tw[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const f32x8 trow = load_frag(sA + r * L::LDA + kb * 32, grp);
      float xu[8], xw[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = kb * 32 + kc(grp, j);
        const float t = trow[j] * sBeta[s];
        xu[j] = t;
        xw[j] = KDA ? t : t * __expf(sGam[s]);
      }
      tu[kb] = make_frag<T>(xu);
      tw[kb] = make_frag<T>(xw);
    }
    // U~ = T Diag(b) V: rows = tokens, columns = d_v; stored transposed [d_v][token]
    T *ut_out = static_cast<T *>(a.Ut) + blk * ((size_t)DV * kChunk);
#pragma unroll
    for (int n = 0; n < DV / 16; ++n) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        acc = mma(acc, tu[kb], load_frag(sVt + (16 * n + col) * L::LDT + kb * 32, grp));
      store4(ut_out + (size_t)(16 * n + col) * kChunk + 16 * i + 4 * grp, acc);
    }
    // W^T = (K e^gamma)^T T'^T: rows = d_k, columns = tokens; stored [token][d_k]
    T *w_out = static_cast<T *>(a.W) + blk * ((size_t)kChunk * DK);
#pragma unroll
    for (int m = 0; m < DK / 16; ++m) {
      const int d = 16 * m + col;
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        Frag<T> kf;
        if constexpr (!KDA) {
          kf = load_frag(sKt + d * L::LDT + kb * 32, grp);
        } else {
          float xk[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int s = kb * 32 + kc(grp, j);
            xk[j] = E::to_f32(sKt[d * L::LDT + s]) * __expf(sGam[s * L::LDG + d]);
          }
          kf = make_frag<T>(xk);
        }
        acc = mma(acc, kf, tw[kb]);
      }
      // rows d = 16m + 4grp + e of this lane, stored negated and kmap-permuted
      // inside their 32-block (logical index (m & 1) * 16 + 4grp + e sits at
      // 8grp + 4(m & 1) + e)
      store4(w_out + (size_t)(16 * i + col) * DK + (m >> 1) * 32 + 8 * grp + 4 * (m & 1), -acc);
    }
  }
}

template <typename T, int DK, int DV, bool KDA>
static hipError_t launch_local_t(const PrefillArgs &a, hipStream_t stream) {
  using L = LocalLayout<T, DK, DV, KDA>;
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&chunk_local_kernel<T, DK, DV, KDA>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)L::bytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((chunk_local_kernel<T, DK, DV, KDA>), dim3(a.max_chunks, a.Hv),
                     dim3(kLocalThreads), L::bytes, stream, a);
  return hipGetLastError();
}

template <typename T, bool KDA>
static hipError_t dispatch_dims(const PrefillArgs &a, hipStream_t s) {
  if (a.Dk == 64 && a.Dv == 64) return launch_local_t<T, 64, 64, KDA>(a, s);
  if (a.Dk == 64 && a.Dv == 128) return launch_local_t<T, 64, 128, KDA>(a, s);
  if (a.Dk == 128 && a.Dv == 64) return launch_local_t<T, 128, 64, KDA>(a, s);
  return launch_local_t<T, 128, 128, KDA>(a, s);
}

hipError_t launch_chunk_local(const PrefillArgs &a, bool bf16, bool kda, hipStream_t s) {
  if (a.max_chunks == 0) return hipSuccess;
  if (bf16) return kda ? dispatch_dims<bf16_t, true>(a, s) : dispatch_dims<bf16_t, false>(a, s);
  return kda ? dispatch_dims<float, true>(a, s) : dispatch_dims<float, false>(a, s);
}

}  // namespace hagdn
