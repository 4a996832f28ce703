// k1_chunk_local.hip -- the first Map phase of chunkwise delta-rule prefill
// (paper Sec. 2.1: operators #1 Gate, #2 KKT, #3 Solve, #4 W/U), one
// workgroup per (chunk, value head), fully parallel over both, plus the
// chunk-local products that let the sequential kernel advance the state with
// a single product per chunk.
//
// For a chunk of n <= 64 tokens (rows >= n are zero-padded, which makes them
// contribute nothing downstream), with gamma the inclusive cumulative
// log-gate inside the chunk (a d_k-vector per token for KDA):
//   #1  gamma_r = sum_{s<=r} g_s
//   #2  A[r][s] = b_r <k_r, e^(gamma_r - gamma_s) k_s>           (s < r)
//       P[r][s] =     <q_r, e^(gamma_r - gamma_s) k_s>           (s <= r)
//   #3  T = (I + A)^-1                       (unit lower triangular, fp32)
//   #4  W  = T Diag(b) (K * e^gamma)         U~ = T Diag(b) V
// With Kt = (K * e^(gamma_last - gamma))^T and D = Diag(e^gamma_last), the
// state update of operator #5 and the output of operator #6 are affine in the
// state S_c entering the chunk (S^T, d_k x d_v):
//   S^T_{c+1} = D S^T_c - M S^T_c + B,        M = Kt W,  B = Kt U~
//   O         = Q' S^T_c + O_loc,             Q' = Q * e^gamma - P W,  O_loc = P U~
// (expand U = U~ - W S^T_c, the corrected values "v_c" of Sec. 5, in
// S^T_{c+1} = D S^T_c + Kt U and O = (Q * e^gamma) S^T_c + P U).  This
// kernel computes the state-independent factors -M, B, Q', O_loc and the
// chunk decay; W and U~ never leave the workgroup.  It is Sec. 5's GEMM-first
// regrouping carried one step further: every product that does not need the
// incoming state runs here, chunk-parallel, so the sequential kernel's
// critical path per chunk is one product.
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
// write the decay; wave i computes token block i of W and U~ into LDS; then
// the four reduce-side products are split over the waves.
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kLocalThreads = 256;

template <typename T, int DK, int DV, bool KDA>
struct LocalLayout {
  static constexpr int PAD = 16 / (int)sizeof(T);
  static constexpr int LDK = DK + PAD;       // sK   [64][LDK]   keys, token rows (ops #2)
  static constexpr int LDT = kChunk + PAD;   // sKt  [DK][LDT]   keys, channel rows
                                             // sVt  [DV][LDT]   values, channel rows (op #4)
                                             // sWt  [DK][LDT]   W, channel rows (over sK)
                                             // sUt  [DV][LDT]   U~, channel rows (over sVt)
  static constexpr int LDA = kChunk + 4;     // sA   [64][LDA]   A, then T (fp32)
  static constexpr int LDG = KDA ? DK + 1 : 1;  // sGam [64][LDG] (GDN: [64])
  static constexpr size_t bytesX = sizeof(T) * (kChunk * LDK > DK * LDT ? kChunk * LDK : DK * LDT);
  static constexpr size_t off_K = 0;         // region X: sK, later sWt
  static constexpr size_t off_Kt = off_K + bytesX;
  static constexpr size_t off_Vt = off_Kt + sizeof(T) * DK * LDT;   // region Y: sVt, later sUt
  static constexpr size_t off_A = off_Vt + sizeof(T) * DV * LDT;
  static constexpr size_t off_beta = off_A + sizeof(float) * kChunk * LDA;
  static constexpr size_t off_kdec = off_beta + sizeof(float) * kChunk;  // GDN e^(gamma_last - gamma_s)
  static constexpr size_t off_gam = off_kdec + sizeof(float) * kChunk;
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
  float *sKdec = reinterpret_cast<float *>(smem + L::off_kdec);
  float *sGam = reinterpret_cast<float *>(smem + L::off_gam);
  T *sWt = sK;   // reuses region X once op #2 is done with the keys
  T *sUt = sVt;  // reuses region Y once op #4 has read the values

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
          Pout[r * kChunk + s] = E::from_f32(vP);
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
          Pout[r * kChunk + sb] = E::from_f32(accP[e]);
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
          Pout[r * kChunk + s] = E::from_f32(s <= r ? accP[e] : 0.f);
        }
      }
      for (int j = i + 1; j < 4; ++j) {  // above the diagonal: zero
        const int s = 16 * j + col;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = r0 + 4 * grp + e;
          sA[r * L::LDA + s] = 0.f;
          Pout[r * kChunk + s] = E::from_f32(0.f);
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
    // chunk decay e^gamma_last, and (GDN) each token's key decay to the chunk end
    const int t2 = tid - 64;
    float *dec_out = a.dec + blk * DK;
    if constexpr (KDA) {
      for (int d = t2; d < DK; d += kLocalThreads - 64)
        dec_out[d] = __expf(sGam[(kChunk - 1) * L::LDG + d]);
    } else {
      if (t2 < kChunk) sKdec[t2] = __expf(sGam[kChunk - 1] - sGam[t2]);
      if (t2 == 0) dec_out[0] = __expf(sGam[kChunk - 1]);
    }
  }
  __syncthreads();

  // ---- op #4: wave i = token block i.  T' = T Diag(b) (GDN: also e^gamma_s).
  // W and U~ go to LDS as channel rows: sWt[d_k][token] (region X, free since
  // op #2), sUt[d_v][token] (region Y, once every wave has read the values).
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
    // U~ rows = tokens, columns = d_v; W rows = tokens, columns = d_k
    f32x4 accU[DV / 16];
#pragma unroll
    for (int n = 0; n < DV / 16; ++n) {
      accU[n] = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        accU[n] = mma(accU[n], tu[kb], load_frag(sVt + (16 * n + col) * L::LDT + kb * 32, grp));
    }
#pragma unroll
    for (int n = 0; n < DK / 16; ++n) {
      const int d = 16 * n + col;
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
        acc = mma(acc, tw[kb], kf);
      }
      // lane: column d, rows (tokens) 16i + 4grp + e
      store4(sWt + d * L::LDT + 16 * i + 4 * grp, acc);
    }
    __syncthreads();  // every wave has read sVt
#pragma unroll
    for (int n = 0; n < DV / 16; ++n) store4(sUt + (16 * n + col) * L::LDT + 16 * i + 4 * grp, accU[n]);
  }
  __syncthreads();

  // ---- reduce-side products.  Kt fragments are built from the staged keys:
  //      Kt[d][s] = K[s][d] e^(gamma_last - gamma_s)  (KDA: per channel d)
  constexpr int KT = DK / 16, VT = DV / 16;
  constexpr int KPW = KT / 4;  // d_k tiles per wave
  auto kt_frag = [&](int d, int kb) {
    float x[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int s = kb * 32 + kc(grp, j);
      const float ex = KDA ? __expf(sGam[(kChunk - 1) * L::LDG + d] - sGam[s * L::LDG + d]) : sKdec[s];
      x[j] = E::to_f32(sKt[d * L::LDT + s]) * ex;
    }
    return make_frag<T>(x);
  };
  {
    // (a) -M = -(Kt W), the state kernel's A operand (fragment order, prefill.h).
    //     Computed transposed, M^T = W^T Kt^T: rows d_in from sWt, columns
    //     d_out from Kt.
    T *nm_out = static_cast<T *>(a.NM) + blk * ((size_t)DK * DK);
#pragma unroll
    for (int nn = 0; nn < KPW; ++nn) {
      const int n = wave * KPW + nn, dout = 16 * n + col;  // this lane's B column
      const Frag<T> bk[2] = {kt_frag(dout, 0), kt_frag(dout, 1)};
#pragma unroll
      for (int m = 0; m < KT; ++m) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          acc = mma(acc, load_frag(sWt + (16 * m + col) * L::LDT + kb * 32, grp), bk[kb]);
        // lane: column d_out, rows d_in = 16m + 4grp + e = 32(m >> 1) + kmap(grp, 4(m & 1) + e)
        // -> slots 4(m & 1) + e of operand block (t = n, kb = m >> 1)
        store4(nm_out + ((size_t)(n * (DK / 32) + (m >> 1)) * 64 + lane) * 8 + 4 * (m & 1), -acc);
      }
    }
    // (b) B = Kt U~, the state kernel's accumulator init (fragment order)
    T *b_out = static_cast<T *>(a.Bc) + blk * ((size_t)DV * DK);
#pragma unroll
    for (int mm = 0; mm < KPW; ++mm) {
      const int m = wave * KPW + mm;
      const Frag<T> ak[2] = {kt_frag(16 * m + col, 0), kt_frag(16 * m + col, 1)};
#pragma unroll
      for (int n = 0; n < VT; ++n) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          acc = mma(acc, ak[kb], load_frag(sUt + (16 * n + col) * L::LDT + kb * 32, grp));
        store4(b_out + ((size_t)(n * (DK / 16) + m) * 64 + lane) * 4, acc);
      }
    }
    // (c) Q' = Q e^gamma - P W and (d) O_loc = P U~, the output kernel's B
    //     operand and accumulator init (fragment order, token tile nt = w);
    //     computed transposed (rows = channels, columns = tokens 16w..16w+15).
    //     P is causal: k-blocks kb <= w/2.
    const int r = 16 * wave + col;
    const T *prow = static_cast<const T *>(a.P) + blk * (kChunk * kChunk) + (size_t)r * kChunk;
    Frag<T> bp[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) bp[kb] = load_frag(prow + kb * 32, grp);
    const int nkb = (wave >> 1) + 1;
    T *qp_out = static_cast<T *>(a.Qp) + blk * ((size_t)kChunk * DK) + (size_t)wave * (DK / 32) * 64 * 8;
    const T *qrow = qbase + (size_t)r * qk_row;
#pragma unroll
    for (int m = 0; m < KT; ++m) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        if (kb < nkb) acc = mma(acc, load_frag(sWt + (16 * m + col) * L::LDT + kb * 32, grp), bp[kb]);
      const int d = 16 * m + 4 * grp;
      f32x4 qe = zero4();
      if (r < len) {
        qe = load4(qrow + d);
#pragma unroll
        for (int e = 0; e < 4; ++e) qe[e] *= KDA ? __expf(sGam[r * L::LDG + d + e]) : __expf(sGam[r]);
      }
      store4(qp_out + ((size_t)(m >> 1) * 64 + lane) * 8 + 4 * (m & 1), qe - acc);
    }
    T *ol_out = static_cast<T *>(a.Ol) + blk * ((size_t)kChunk * DV) + (size_t)wave * (DV / 16) * 64 * 4;
#pragma unroll
    for (int m = 0; m < VT; ++m) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        if (kb < nkb) acc = mma(acc, load_frag(sUt + (16 * m + col) * L::LDT + kb * 32, grp), bp[kb]);
      store4(ol_out + ((size_t)m * 64 + lane) * 4, acc);
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
