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
// sits inside the contraction: every 16x16 block of row block i factors it
// around the token rho = 16i + 8 in the middle of the block,
// <k_r e^(gamma_r - gamma_rho), k_s e^(gamma_rho - gamma_s)>; inside the block
// each factor spans at most 8 tokens of decay, off-diagonal s-side factors are
// <= 1, and upper-triangle products (which may overflow) are discarded by
// selection.
//
// Wave roles (4 waves): wave i computes row block i of A and P; wave 0 then
// solves T by forward substitution (lane j owns column j) while waves 1-3
// write the decay; wave i computes token block i of W and U~ into LDS; then
// the four reduce-side products are split over the waves.
#include <algorithm>
#include <atomic>

#include "device.h"
#include "prefill.h"
#include "state_walk.h"

namespace hagdn {

constexpr int kLocalThreads = 256;

// XOR-swizzled row-major tiles (rows of LD elements, a multiple of 128 bytes):
// 16-byte chunk q of row r is stored at chunk q ^ (r & 7), so the eight rows
// a fragment read touches in one LDS cycle hit eight different bank groups
// with no padding.
template <typename E, int LD>
__device__ __forceinline__ int swz(int r, int e) {
  constexpr int CH = 16 / (int)sizeof(E);
  return r * LD + ((e / CH) ^ (r & 7)) * CH + e % CH;
}
// MFMA fragment: the 8 elements at logical columns e .. e+7 (e a multiple of 8) of row r.
template <int LD>
__device__ __forceinline__ bf16x8 frag_sw(const bf16_t *t, int r, int e) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(t + swz<bf16_t, LD>(r, e)));
}
template <int LD>
__device__ __forceinline__ f32x8 frag_sw(const float *t, int r, int e) {
  const f32x4 x = *reinterpret_cast<const f32x4 *>(t + swz<float, LD>(r, e));
  const f32x4 y = *reinterpret_cast<const f32x4 *>(t + swz<float, LD>(r, e + 4));
  return __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Three tile regions, each reused once its first tenant is dead:
//   X  sK  [64][DK]  keys, token rows (op #2)   -> sKt [DK][64] keys, channel rows (op #4 on)
//   Y  sA  [64][64]  A, then T (fp32, ops #2-#3) -> sWt [DK][64] W, channel rows
//   Z  sVt [DV][64]  values, channel rows         -> sUt [DV][64] U~, channel rows
// all XOR-swizzled; plus the gate scan gamma.  GDN also keeps beta and its
// decay column e^(gamma_last - gamma_s) here.  KDA's gamma is a [64][DK]
// table, so a KDA item holds beta in registers and runs its gate-scan totals
// through region Y (free until op #2): at d_k = d_v = 128, bf16, that keeps
// the item at exactly 80 KiB, two per CU.
template <typename T, int DK, int DV, bool KDA>
struct LocalLayout {
  static constexpr int LDK = DK;       // sK row length
  static constexpr int LDT = kChunk;   // channel-row length (sKt, sWt, sVt, sUt)
  static constexpr int LDA = kChunk;   // sA row length
  static constexpr size_t bytesX = sizeof(T) * kChunk * DK;
  static constexpr size_t bytesY = sizeof(float) * kChunk * kChunk > sizeof(T) * DK * kChunk
                                       ? sizeof(float) * kChunk * kChunk : sizeof(T) * DK * kChunk;
  static constexpr size_t off_K = 0;   // region X
  static constexpr size_t off_A = off_K + bytesX;   // region Y
  static constexpr size_t off_Vt = off_A + bytesY;  // region Z
  static constexpr size_t off_beta = off_Vt + sizeof(T) * DV * kChunk;                // GDN
  static constexpr size_t off_kdec = off_beta + (KDA ? 0 : sizeof(float) * kChunk);   // GDN
  static constexpr size_t off_gam = off_kdec + (KDA ? 0 : sizeof(float) * kChunk);
  // GDN: the scalar gate scan in fp64 (gamma reaches thousands in magnitude
  // where gates are near 0, and the decays are exponentials of differences)
  static constexpr size_t bytes = off_gam + (KDA ? sizeof(float) * kChunk * DK : sizeof(double) * kChunk);
  // KDA gate-scan segment totals: kLocalThreads floats in region Y, behind the
  // kLocalThreads-float scratch of the q/k normalisation
  static constexpr size_t off_tot = off_A + sizeof(float) * kLocalThreads;
  static_assert(!KDA || off_tot + sizeof(float) * kLocalThreads <= off_A + bytesY, "totals fit region Y");
};

// KDA gamma[r][d] in the [64][DK] table, rows unpadded: the 16-byte chunk q of
// row r is stored at chunk q ^ f(r), f(r) = (r & 7) ^ 4 ((r >> 3) & 1).  The
// (r & 7) term lets eight consecutive token rows read the same channels as
// 16-byte vectors with no bank conflict (op #2, Q'); the second term puts
// token rows 8 apart into different halves of a 32-channel block, so the
// per-element reads of op #4 (16 channels x 4 token rows 8 apart) conflict at
// most 2-way.  Chunks move only inside their 32-channel block.
template <int DK>
__device__ __forceinline__ int gam_at(int r, int d) {
  const int f = (r & 7) ^ (((r >> 3) & 1) << 2);
  return r * DK + ((((d >> 2) ^ f) << 2) | (d & 3));
}
// gamma[r][d .. d+7] (d a multiple of 8) as two 16-byte reads
template <int DK>
__device__ __forceinline__ void gam8(const float *g, int r, int d, float (&x)[8]) {
  const f32x4 lo = *reinterpret_cast<const f32x4 *>(g + gam_at<DK>(r, d));
  const f32x4 hi = *reinterpret_cast<const f32x4 *>(g + gam_at<DK>(r, d + 4));
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[e] = lo[e];
    x[4 + e] = hi[e];
  }
}

// One (chunk, value head) work item: chunk c = item / Hv, head h = item % Hv.
struct LocalItem {
  int c, h, start, len;  // len 0: past the last chunk
};
// Workgroup b -> item: the value heads of one q/k group (grouped heads share
// q and k) take consecutive ids of one XCD (ids b, b+8, ... share an XCD and
// its L2), so all but the first read q and k from L2.  Without grouping this
// is the identity.  The grid is padded to whole rounds of 8 groups.
__device__ __forceinline__ LocalItem local_item(const PrefillArgs &a, int b) {
  LocalItem it{0, 0, 0, 0};
  const int G = a.Hv / a.Hqk;  // value heads per q/k head
  const int xcd = b % 8, slot = b / 8;
  const int grp = (slot / G) * 8 + xcd;  // (chunk, q/k head) group
  if (grp < a.max_chunks * a.Hqk) {
    it.c = grp / a.Hqk;
    it.h = (grp % a.Hqk) * G + slot % G;
    if (a.single) {  // chunk c of the only sequence (tokens [0, T))
      it.start = it.c * kChunk;
      it.len = max(0, min(kChunk, a.T - it.start));
    } else {
      const int4 ci = a.chunk_info[it.c];
      it.start = ci.y;
      it.len = ci.z;
    }
  }
  return it;
}

// Overlapped launch: the next item of this XCD's queue.  XCD x serves the
// value heads h = x (mod 8) (ovl_heads), chunk-major, so the blocks of a head
// are produced in chunk order on the XCD whose L2 that head's walks read.
__device__ __forceinline__ LocalItem ovl_item(const PrefillArgs &a) {
  __shared__ int ticket;
  const int x = xcc_id();
  if (threadIdx.x == 0) ticket = atomicAdd(a.ovl + kOvlLocalQ + kOvlStride * x, 1);
  __syncthreads();
  const int t = ticket;
  const int hx = ovl_heads(a.Hv, x);
  LocalItem it{0, 0, 0, 0};
  if (hx > 0 && t < a.max_chunks * hx) {
    it.c = t / hx;
    it.h = x + kXcdCount * (t % hx);
    if (a.single) {
      it.start = it.c * kChunk;
      it.len = max(0, min(kChunk, a.T - it.start));
    } else {
      const int4 ci = a.chunk_info[it.c];
      it.start = ci.y;
      it.len = ci.z;
    }
  }
  return it;
}

// Overlapped launch, walk role: the next whole-chain walk tile of this XCD's
// queue (value heads h = x (mod 8), every sequence, every d_v tile).
template <typename T, int DK, int DV, bool KDA, bool SINGLE>
__device__ __forceinline__ void ovl_walk(const PrefillArgs &a) {
  constexpr int NT = DV / 16;
  __shared__ int ticket;
  const int x = xcc_id();
  const int hx = ovl_heads(a.Hv, x);
  // A walker takes tiles until its XCD's queue is empty: the grid gives every
  // XCD its share and two more, and should a dispatch deal the grid unevenly,
  // the walkers that did land on an XCD still walk all of its tiles.
  for (;;) {
    if (threadIdx.x == 0) ticket = atomicAdd(a.ovl + kOvlWalkQ + kOvlStride * x, 1);
    __syncthreads();
    const int t = ticket;
    __syncthreads();  // every wave has read the ticket before the next one is taken
    if (hx == 0 || t >= a.N * hx * NT) return;  // uniform for the workgroup
    const int j = t / NT, n = j / hx, h = x + kXcdCount * (j % hx);
    walk_tile<T, DK, DV, KDA, SINGLE, true>(a, n * a.Hv + h, t % NT);
    __syncthreads();  // the walk's exchange buffer is free again
  }
}

// Global inputs of one item (padded tokens: zeros).
// Every load is issued unconditionally from a row clamped into the chunk and
// the padding is selected away afterwards, so the memory counters stay exact.
template <typename T, int DK, int DV, bool KDA, bool PRE>
struct LocalIn {
  static constexpr int V = 16 / (int)sizeof(T);
  static constexpr int NKV = DK / 4 / V, NVV = DV / 4 / V;       // 16-byte vectors per lane
  static constexpr int GPT = KDA ? kChunk * DK / kLocalThreads : 1;  // gate values per thread
  u32x4 kv[NKV], vv[NVV];  // keys, values: lane = token, wave = channel quarter
  float bval, gk[GPT];     // beta of token tid (KDA: of token 16 wave + col); gates (KDA: thread = (channel, token segment))
  Frag<T> qf[DK / 32];     // queries of token 16 wave + col, op #2 operand
  f32x4 qacc[DK / 16];     // the same queries in accumulator layout (channels 16m + 4grp ..)

  __device__ __forceinline__ void load_kvg(const PrefillArgs &a, const LocalItem &it) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int hk = it.h / (a.Hv / a.Hqk);
    const int last = it.len - 1;
    const size_t qk_row = (size_t)a.Hqk * DK, v_row = (size_t)a.Hv * DV;
    const int rk = min(lane, last);
    const T *kb = static_cast<const T *>(a.k) + (size_t)(it.start + rk) * qk_row + (size_t)hk * DK + wave * (DK / 4);
    const T *vb = static_cast<const T *>(a.v) + (size_t)(it.start + rk) * v_row + (size_t)it.h * DV + wave * (DV / 4);
    const bool live = lane < it.len;
#pragma unroll
    for (int i = 0; i < NKV; ++i) {
      const u32x4 x = *reinterpret_cast<const u32x4 *>(kb + i * V);
      kv[i] = live ? x : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < NVV; ++i) {
      const u32x4 x = *reinterpret_cast<const u32x4 *>(vb + i * V);
      vv[i] = live ? x : u32x4{0, 0, 0, 0};
    }
    // GDN: thread tid < 64 holds beta of token tid (staged in LDS); KDA: each
    // lane holds beta of its op #2 token 16 wave + col
    const int bt = KDA ? 16 * wave + (lane & 15) : tid;
    const float b = a.beta[(size_t)(it.start + min(bt & (kChunk - 1), last)) * a.Hv + it.h];
    const float bx = (PRE && (a.pre & kPreBetaSigmoid)) ? sigmoid(b) : b;
    bval = (bt < kChunk && bt < it.len) ? bx : 0.f;
    const int rt = min(tid & (kChunk - 1), last);
    if constexpr (KDA) {
      const int d = tid % DK, seg = tid / DK;
      const float *gb = a.g + ((size_t)it.start * a.Hv + it.h) * DK + d;
#pragma unroll
      for (int u = 0; u < GPT; ++u) {
        const int r = seg * GPT + u;
        const float x = gb[(size_t)min(r, last) * a.Hv * DK];
        gk[u] = r < it.len ? ((PRE && (a.pre & kPreGateSoftplus)) ? neg_softplus(x) : x) : 0.f;
      }
    } else {
      const float x = a.g[(size_t)(it.start + rt) * a.Hv + it.h];
      const float gx = (PRE && (a.pre & kPreGateSoftplus)) ? neg_softplus(x) : x;
      gk[0] = (tid < kChunk && tid < it.len) ? gx : 0.f;
    }
  }
  __device__ __forceinline__ void load_q(const PrefillArgs &a, const LocalItem &it) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int col = lane & 15, grp = lane >> 4;
    const int rq = 16 * wave + col;
    const int hk = it.h / (a.Hv / a.Hqk);
    const size_t qk_row = (size_t)a.Hqk * DK;
    const T *qrow = static_cast<const T *>(a.q) + (size_t)(it.start + min(rq, it.len - 1)) * qk_row + (size_t)hk * DK;
    const bool live = rq < it.len;
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) {
      const Frag<T> x = load_frag(qrow + kb * 32, grp);
      qf[kb] = live ? x : zero_frag<T>();
    }
#pragma unroll
    for (int m = 0; m < DK / 16; ++m) {
      const f32x4 x = load4(qrow + 16 * m + 4 * grp);
      qacc[m] = live ? x : zero4();
    }
  }
  // L2 normalisation of raw keys and queries.  A key row is spread over the
  // four waves (channel quarters): their partial sums of squares meet in
  // `scratch` (256 floats, one barrier) and the keys are rescaled in
  // registers before they are staged.  A query row lives in the four lane
  // groups of one column (two lane exchanges); its factor is applied to the
  // products the queries enter (P and Q * e^gamma), which is the same as
  // scaling the query rows, and is formed only when op #2 needs it, so the
  // query loads are waited for no earlier.
  __device__ __forceinline__ void l2norm_k(float *scratch) {
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    using V16 = Vec16<T>;
    float ss = 0.f;
#pragma unroll
    for (int i = 0; i < NKV; ++i) {
      const uint4 u = __builtin_bit_cast(uint4, kv[i]);
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const float x = V16::get(u, j);
        ss += x * x;
      }
    }
    scratch[wave * 64 + lane] = ss;
    __syncthreads();
    const float ik = inv_l2(scratch[lane] + scratch[64 + lane] + scratch[128 + lane] + scratch[192 + lane]);
#pragma unroll
    for (int i = 0; i < NKV; ++i) {
      const uint4 u = __builtin_bit_cast(uint4, kv[i]);
      float x[V];
#pragma unroll
      for (int j = 0; j < V; ++j) x[j] = V16::get(u, j) * ik;
      kv[i] = __builtin_bit_cast(u32x4, V16::pack(x));
    }
  }
  __device__ __forceinline__ float l2norm_q() const {
    float qs = 0.f;
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const float x = frag_elem(qf[kb], j);
        qs += x * x;
      }
    qs += __shfl_xor(qs, 16);
    qs += __shfl_xor(qs, 32);
    return inv_l2(qs);
  }
};

// PRE: the call carries preprocessing flags (a separate instance, so that the
// plain path keeps its register budget).  OVL: the overlapped launch (1: a
// single sequence, 2: a batch): every workgroup takes a chunk-local item from
// its XCD's queue and publishes the block's ready flag once its factors are
// stored; workgroups below a.ovl_walk_wgs then walk a whole chain
// (ovl_walk).
template <typename T, int DK, int DV, bool KDA, bool PRE, int OVL = 0>
__global__ __launch_bounds__(kLocalThreads, OVL || (KDA && sizeof(T) == 2) ? 2 : 1) void chunk_local_kernel(PrefillArgs a) {
  using L = LocalLayout<T, DK, DV, KDA>;
  using V16 = Vec16<T>;
  using In = LocalIn<T, DK, DV, KDA, PRE>;
  constexpr int V = 16 / (int)sizeof(T);  // elements per 16-byte vector
  constexpr int KT = DK / 16, VT = DV / 16;
  constexpr int KPW = KT / 4;             // d_k tiles per wave in the reduce-side products
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  // overlapped launch: walk workgroups also produce one chunk-local item
  // first, while the first chunks are being computed everywhere
  const bool walker = OVL != 0 && (int)blockIdx.x < a.ovl_walk_wgs;
  const LocalItem cur = OVL ? ovl_item(a) : local_item(a, blockIdx.x);
  if (cur.len <= 0) {  // past the last chunk: uniform for the workgroup
    if constexpr (OVL != 0) {
      if (walker) ovl_walk<T, DK, DV, KDA, OVL == 1>(a);
    }
    return;
  }
  In in;
  in.load_kvg(a, cur);
  in.load_q(a, cur);
  const int c = cur.c, h = cur.h, start = cur.start, len = cur.len;
  const size_t blk = (size_t)c * a.Hv + h;

  extern __shared__ __align__(16) unsigned char smem[];
  T *sK = reinterpret_cast<T *>(smem + L::off_K);
  T *sKt = sK;   // region X once op #2 is done with the token rows
  T *sVt = reinterpret_cast<T *>(smem + L::off_Vt);
  float *sA = reinterpret_cast<float *>(smem + L::off_A);
  float *sBeta = reinterpret_cast<float *>(smem + L::off_beta);
  float *sKdec = reinterpret_cast<float *>(smem + L::off_kdec);
  float *sTot = reinterpret_cast<float *>(smem + L::off_tot);
  float *sGam = reinterpret_cast<float *>(smem + L::off_gam);     // KDA: [64][DK] (gam_at)
  double *sGd = reinterpret_cast<double *>(smem + L::off_gam);    // GDN: [64], fp64
  T *sWt = reinterpret_cast<T *>(smem + L::off_A);  // region Y once every wave holds its T rows
  T *sUt = sVt;  // region Z once op #4 has read the values

  const int rq = 16 * wave + col;  // token this lane feeds as a column of A^T and P^T
  constexpr int NKV = In::NKV, NVV = In::NVV, GPT = In::GPT;
  const u32x4(&kv)[NKV] = in.kv;
  const u32x4(&vv)[NVV] = in.vv;
  const Frag<T>(&qf)[DK / 32] = in.qf;
  const f32x4(&qacc)[KT] = in.qacc;
  float(&gk)[GPT] = in.gk;
  const float bval = in.bval;

  // raw projections: normalise q and k (region Y is free until op #2)
  float qscale = 1.f;  // L2 factor of this lane's query row rq (raw queries), set before op #2
  if constexpr (PRE) {
    if (a.pre & kPreQkNorm) in.l2norm_k(sA);
  }

  // ---- stage K (token rows; its channel rows follow op #2 in the same
  //      region) and V (channel rows); the channel-row writes of one wave
  //      cover 64 consecutive tokens of one row
#pragma unroll
  for (int it = 0; it < NKV; ++it) {
    const int cv = wave * (DK / 4) + it * V;
    *reinterpret_cast<u32x4 *>(sK + swz<T, L::LDK>(lane, cv)) = kv[it];
  }
#pragma unroll
  for (int it = 0; it < NVV; ++it) {
    const int cv = wave * (DV / 4) + it * V;
    const uint4 u = __builtin_bit_cast(uint4, vv[it]);
#pragma unroll
    for (int j = 0; j < V; ++j) sVt[swz<T, L::LDT>(cv + j, lane)] = V16::raw(u, j);
  }
  // ---- op #1: beta and gamma (inclusive cumulative log-gate)
  if constexpr (!KDA) {
    if (tid < kChunk) sBeta[tid] = bval;
  }
  if constexpr (!KDA) {
    if (wave == 0) {
      double x = gk[0];
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const double y = __shfl_up(x, off);
        if (lane >= off) x += y;
      }
      sGd[lane] = x;
    }
  } else {
    // segment-local scan in registers, then add the totals of earlier segments
    const int d = tid % DK, seg = tid / DK;
#pragma unroll
    for (int u = 1; u < GPT; ++u) gk[u] += gk[u - 1];
    sTot[seg * DK + d] = gk[GPT - 1];
    __syncthreads();
    float off = 0.f;
    for (int s2 = 0; s2 < seg; ++s2) off += sTot[s2 * DK + d];
#pragma unroll
    for (int u = 0; u < GPT; ++u) sGam[gam_at<DK>(seg * GPT + u, d)] = gk[u] + off;
  }
  __syncthreads();

  // ---- op #2, transposed: wave i owns tokens r in [16i, 16i+16) as the
  //      columns of A^T and P^T and computes the row blocks s = 16j.. (j <= i).
  //      A goes to LDS row-major (A[r][s], 4 consecutive s per lane); the P^T
  //      accumulators stay in registers: two of them form the P^T fragment of
  //      a 32-token k-block (accumulator slot map), the B operand of Q' and O_loc.
  if constexpr (PRE) {
    if (a.pre & kPreQkNorm) qscale = in.l2norm_q();
  }
  f32x4 accP[4];
  {
    const int i = wave, r = rq;
    f32x4 accA[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) accA[j] = accP[j] = zero4();
    if constexpr (!KDA) {
      Frag<T> kr[DK / 32];
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb) kr[kb] = frag_sw<L::LDK>(sK, r, kb * 32 + 8 * grp);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if (j <= i) {
#pragma unroll
          for (int kb = 0; kb < DK / 32; ++kb) {
            const Frag<T> ks = frag_sw<L::LDK>(sK, 16 * j + col, kb * 32 + 8 * grp);
            accA[j] = mma(accA[j], ks, kr[kb]);
            accP[j] = mma(accP[j], ks, qf[kb]);
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int s = 16 * j + 4 * grp + e;
          const float dec = s <= r ? __expf((float)(sGd[r] - sGd[s])) : 0.f;
          accA[j][e] = s < r ? sBeta[r] * accA[j][e] * dec : 0.f;
          accP[j][e] = accP[j][e] * dec * qscale;
        }
        *reinterpret_cast<f32x4 *>(sA + swz<float, L::LDA>(r, 16 * j + 4 * grp)) = accA[j];
      }
    } else {
      // Per-channel decay e^(gamma_r - gamma_s), factored around a reference
      // token rho in the middle of this wave's block: the r side carries
      // e^(gamma_r - gamma_rho), the s side e^(gamma_rho - gamma_s), so every
      // block -- the diagonal one included -- is an MFMA product.  Inside the
      // block each factor spans at most 8 tokens of decay; off-diagonal s-side
      // factors are <= 1.  Upper-triangle products of the diagonal block may
      // overflow: they are discarded by selection below, never multiplied.
      //
      // This is exact up to rounding while every exponent of the block stays
      // within +-kFactorExp (kFactorExp < 88, the fp32/bf16 overflow point):
      // no factor overflows, and an s-side factor that underflows belongs to
      // a product below e^(kFactorExp - 87), far under any rounding error.  A
      // block in which some channel decays by more than e^kFactorExp over
      // half a block (a strongly forgetting channel: a gate near 0 for a few
      // tokens) takes the exact path instead: off-diagonal blocks factored
      // around the last token of the s block (both factors <= 1), the diagonal
      // block elementwise.  The choice is per wave (one row block), uniform.
      constexpr float kFactorExp = 40.f;
      const int rho = 16 * i + 8;
      bool wide = false;
#pragma unroll
      for (int kb = 0; kb < DK / 32; ++kb) {
        float gr[8], gh[8];
        gam8<DK>(sGam, r, kb * 32 + kc(grp, 0), gr);
        gam8<DK>(sGam, rho, kb * 32 + kc(grp, 0), gh);
#pragma unroll
        for (int jj = 0; jj < 8; ++jj) wide |= fabsf(gr[jj] - gh[jj]) > kFactorExp;
      }
      if (!__builtin_amdgcn_ballot_w64(wide)) {
        // B operands (token r side): k_r e^(gamma_r - gamma_rho), q_r e^(gamma_r - gamma_rho)
        Frag<T> kr[DK / 32], qr[DK / 32];
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb) {
          float xk[8], xq[8], gr[8], gh[8];
          const Frag<T> kraw = frag_sw<L::LDK>(sK, r, kb * 32 + 8 * grp);  // channels kc(grp, 0..7)
          gam8<DK>(sGam, r, kb * 32 + kc(grp, 0), gr);
          gam8<DK>(sGam, rho, kb * 32 + kc(grp, 0), gh);
#pragma unroll
          for (int jj = 0; jj < 8; ++jj) {
            const float ex = __expf(gr[jj] - gh[jj]);
            xk[jj] = frag_elem(kraw, jj) * ex;
            xq[jj] = frag_elem(qf[kb], jj) * ex;
          }
          kr[kb] = make_frag<T>(xk);
          qr[kb] = make_frag<T>(xq);
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (j <= i) {  // uniform for the wave
            const int sb = 16 * j + col;
#pragma unroll
            for (int kb = 0; kb < DK / 32; ++kb) {
              float xs[8], gh[8], gs[8];
              const Frag<T> sraw = frag_sw<L::LDK>(sK, sb, kb * 32 + 8 * grp);
              gam8<DK>(sGam, rho, kb * 32 + kc(grp, 0), gh);
              gam8<DK>(sGam, sb, kb * 32 + kc(grp, 0), gs);
#pragma unroll
              for (int jj = 0; jj < 8; ++jj) xs[jj] = frag_elem(sraw, jj) * __expf(gh[jj] - gs[jj]);
              const Frag<T> ks = make_frag<T>(xs);
              accA[j] = mma(accA[j], ks, kr[kb]);
              accP[j] = mma(accP[j], ks, qr[kb]);
            }
          }
        }
      } else {
        // off-diagonal blocks j < i around the last token e of block j:
        // e^(gamma_r - gamma_e) <= 1 (r > e) and e^(gamma_e - gamma_s) <= 1 (s <= e)
#pragma unroll
        for (int j = 0; j < 3; ++j) {
          if (j < i) {  // uniform for the wave
            const int e = 16 * j + 15, sb = 16 * j + col;
#pragma unroll
            for (int kb = 0; kb < DK / 32; ++kb) {
              float xk[8], xq[8], xs[8], gr[8], ge[8], gs[8];
              const Frag<T> kraw = frag_sw<L::LDK>(sK, r, kb * 32 + 8 * grp);
              const Frag<T> sraw = frag_sw<L::LDK>(sK, sb, kb * 32 + 8 * grp);
              gam8<DK>(sGam, r, kb * 32 + kc(grp, 0), gr);
              gam8<DK>(sGam, e, kb * 32 + kc(grp, 0), ge);
              gam8<DK>(sGam, sb, kb * 32 + kc(grp, 0), gs);
#pragma unroll
              for (int jj = 0; jj < 8; ++jj) {
                const float fr = __expf(gr[jj] - ge[jj]);
                xk[jj] = frag_elem(kraw, jj) * fr;
                xq[jj] = frag_elem(qf[kb], jj) * fr;
                xs[jj] = frag_elem(sraw, jj) * __expf(ge[jj] - gs[jj]);
              }
              const Frag<T> ks = make_frag<T>(xs);
              accA[j] = mma(accA[j], ks, make_frag<T>(xk));
              accP[j] = mma(accP[j], ks, make_frag<T>(xq));
              __builtin_amdgcn_sched_barrier(0);
            }
          }
        }
        // diagonal block elementwise in fp32, one token s = 16i + sl at a time:
        // lane (col, grp) sums its 32 channels for token r = 16i + col (with
        // e^min(gamma_r - gamma_s, 0): upper-triangle terms, s > r, are
        // discarded below), the four lane groups of a column add up, and the
        // lane group that holds accumulator row s keeps the sum
        f32x4 va = zero4(), vp = zero4();
#pragma unroll 1
        for (int sl = 0; sl < 16; ++sl) {
          float sa = 0.f, sp = 0.f;
#pragma unroll
          for (int kb = 0; kb < DK / 32; ++kb) {
            float gr[8], gs[8];
            const Frag<T> kraw = frag_sw<L::LDK>(sK, r, kb * 32 + 8 * grp);
            const Frag<T> sraw = frag_sw<L::LDK>(sK, 16 * i + sl, kb * 32 + 8 * grp);
            gam8<DK>(sGam, r, kb * 32 + kc(grp, 0), gr);
            gam8<DK>(sGam, 16 * i + sl, kb * 32 + kc(grp, 0), gs);
#pragma unroll
            for (int jj = 0; jj < 8; ++jj) {
              const float t = frag_elem(sraw, jj) * __expf(fminf(gr[jj] - gs[jj], 0.f));
              sa += frag_elem(kraw, jj) * t;
              sp += frag_elem(qf[kb], jj) * t;
            }
            __builtin_amdgcn_sched_barrier(0);  // one k-block of operands in registers at a time
          }
          sa += __shfl_xor(sa, 16);
          sa += __shfl_xor(sa, 32);
          sp += __shfl_xor(sp, 16);
          sp += __shfl_xor(sp, 32);
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const bool mine = 4 * grp + e == sl;
            va[e] = mine ? sa : va[e];
            vp[e] = mine ? sp : vp[e];
          }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (j == i) {  // uniform for the wave
            accA[j] = va;
            accP[j] = vp;
          }
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int s = 16 * j + 4 * grp + e;
          accA[j][e] = (j <= i && s < r) ? bval * accA[j][e] : 0.f;  // bval: beta of token r
          accP[j][e] = (j <= i && s <= r) ? accP[j][e] * qscale : 0.f;
        }
        *reinterpret_cast<f32x4 *>(sA + swz<float, L::LDA>(r, 16 * j + 4 * grp)) = accA[j];
      }
    }
  }
  __syncthreads();
  // KDA: beta of the tokens this lane scales T's columns by in op #4 (no LDS
  // copy: the gate table fills it); loaded here, used after the solve
  float bs[KDA ? 2 : 1][8];
  if constexpr (KDA) {
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = kb * 32 + kc(grp, j);
        const float b = a.beta[(size_t)(start + min(s, len - 1)) * a.Hv + h];
        const float bx = (PRE && (a.pre & kPreBetaSigmoid)) ? sigmoid(b) : b;
        bs[kb][j] = s < len ? bx : 0.f;
      }
  }
  // keys as channel rows over the token rows op #2 is done with (region X)
#pragma unroll
  for (int it = 0; it < NKV; ++it) {
    const int cv = wave * (DK / 4) + it * V;
    const uint4 u = __builtin_bit_cast(uint4, kv[it]);
#pragma unroll
    for (int j = 0; j < V; ++j) sKt[swz<T, L::LDT>(cv + j, lane)] = V16::raw(u, j);
  }

  // ---- op #3: T = (I + A)^-1 (unit lower triangular, fp32), blocked by 16.
  //      Diagonal blocks: wave w inverts block w by forward substitution (lane
  //      j < 16 solves column j).  Then block rows i = 1..3: wave j < i forms
  //      T_ij = -T_ii sum_{k=j}^{i-1} A_ik T_kj with fp32 MFMA (16x16x4), and
  //      block row i overwrites A's block row i, which later rows never read.
  if (lane < 16) {
    const int b0 = 16 * wave, j = lane;
    float x[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float acc = (r == j) ? 1.f : 0.f;
#pragma unroll
      for (int s = 0; s < r; ++s) acc -= sA[swz<float, L::LDA>(b0 + r, b0 + s)] * x[s];
      x[r] = acc;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) sA[swz<float, L::LDA>(b0 + r, b0 + j)] = x[r];
  }
  __syncthreads();
#pragma unroll
  for (int i = 1; i < 4; ++i) {
    f32x4 res = zero4();
    if (wave < i) {
      const int j = wave;
      f32x4 y = zero4();  // sum_k A_ik T_kj
      for (int k = j; k < i; ++k) {
#pragma unroll
        for (int st = 0; st < 4; ++st) {
          const float av = sA[swz<float, L::LDA>(16 * i + col, 16 * k + 4 * st + grp)];
          const float tv = sA[swz<float, L::LDA>(16 * k + 4 * st + grp, 16 * j + col)];
          y = __builtin_amdgcn_mfma_f32_16x16x4f32(av, tv, y, 0, 0, 0);
        }
      }
      // T_ii y: the accumulator rows 4grp + st of y are the k index of step st
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const float tv = sA[swz<float, L::LDA>(16 * i + col, 16 * i + 4 * grp + st)];
        res = __builtin_amdgcn_mfma_f32_16x16x4f32(tv, y[st], res, 0, 0, 0);
      }
    }
    __syncthreads();  // every read of block row i of A is done
    if (wave < i) {
#pragma unroll
      for (int e = 0; e < 4; ++e) sA[swz<float, L::LDA>(16 * i + 4 * grp + e, 16 * wave + col)] = -res[e];
    }
    __syncthreads();
  }

  // ---- op #4: wave i = token block i.  T' = T Diag(b) (GDN: also e^gamma_s).
  //      W and U~ go to LDS as channel rows with tokens kmap-permuted inside
  //      each 32-token block: sWt[d_k][.] over T (region Y) once every wave
  //      holds its T rows, sUt[d_v][.] over the values once every wave has
  //      read them.
  {
    const int i = wave, r = 16 * i + col;
    if constexpr (!KDA) {
      if (tid < kChunk) sKdec[tid] = __expf((float)(sGd[kChunk - 1] - sGd[tid]));
    }
    Frag<T> tu[2], tw[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const f32x8 trow = frag_sw<L::LDA>(sA, r, kb * 32 + 8 * grp);
      float xu[8], xw[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int s = kb * 32 + kc(grp, j);
        const float t = trow[j] * (KDA ? bs[kb][j] : sBeta[s]);
        xu[j] = t;
        xw[j] = KDA ? t : t * __expf((float)sGd[s]);
      }
      tu[kb] = make_frag<T>(xu);
      tw[kb] = make_frag<T>(xw);
    }
    __syncthreads();  // T is in registers: region Y takes W
    f32x4 accU[VT];
#pragma unroll
    for (int n = 0; n < VT; ++n) {
      accU[n] = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        accU[n] = mma(accU[n], tu[kb], frag_sw<L::LDT>(sVt, 16 * n + col, kb * 32 + 8 * grp));
    }
    // lane rows are tokens 16i + 4grp + e: slots 4(i & 1) + e of k-block i >> 1
    const int tpos = 32 * (i >> 1) + 8 * grp + 4 * (i & 1);
#pragma unroll
    for (int n = 0; n < KT; ++n) {
      const int d = 16 * n + col;
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        Frag<T> kf;
        if constexpr (!KDA) {
          kf = frag_sw<L::LDT>(sKt, d, kb * 32 + 8 * grp);
        } else {
          float xk[8];
          const Frag<T> kraw = frag_sw<L::LDT>(sKt, d, kb * 32 + 8 * grp);  // tokens kc(grp, 0..7)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int s = kb * 32 + kc(grp, j);
            xk[j] = frag_elem(kraw, j) * __expf(sGam[gam_at<DK>(s, d)]);
          }
          kf = make_frag<T>(xk);
        }
        acc = mma(acc, tw[kb], kf);
      }
      store4(sWt + swz<T, L::LDT>(d, tpos), acc);
    }
    __syncthreads();  // every wave has read sVt and sKt
#pragma unroll
    for (int n = 0; n < VT; ++n) store4(sUt + swz<T, L::LDT>(16 * n + col, tpos), accU[n]);
  }
  // ---- Kt = (K * e^(gamma_last - gamma))^T in place of the staged keys, tokens
  //      kmap-permuted like sWt / sUt (kmap moves tokens only inside their
  //      32-token block).  Thread tid < 2 DK takes channel row tid % DK and
  //      32-token block tid / DK, so at d_k = 128 all four waves share it.
  if (tid < DK * (kChunk / 32)) {
    constexpr int UH = 32 / V;  // 16-byte vectors per 32-token block
    const int d = tid % DK, base = 32 * (tid / DK);
    uint4 row[UH];
#pragma unroll
    for (int u = 0; u < UH; ++u) row[u] = *reinterpret_cast<const uint4 *>(sKt + swz<T, L::LDT>(d, base + u * V));
#pragma unroll
    for (int u = 0; u < UH; ++u) {
      float outv[V];
#pragma unroll
      for (int j = 0; j < V; ++j) {
        const int p = u * V + j;            // position inside the 32-token block
        const int s = kmap(p >> 3, p & 7);  // token held there, relative to base
        const float ex = KDA ? __expf(sGam[gam_at<DK>(kChunk - 1, d)] - sGam[gam_at<DK>(base + s, d)])
                             : sKdec[base + s];
        outv[j] = V16::get(row[s / V], s % V) * ex;
      }
      *reinterpret_cast<uint4 *>(sKt + swz<T, L::LDT>(d, base + u * V)) = V16::pack(outv);
    }
  }
  {  // chunk decay e^gamma_last
    float *dec_out = a.dec + blk * DK;
    if constexpr (KDA) {
      if (tid < DK) dec_out[tid] = __expf(sGam[gam_at<DK>(kChunk - 1, tid)]);
    } else {
      if (tid == 0) dec_out[0] = __expf((float)sGd[kChunk - 1]);
    }
  }
  __syncthreads();

  // ---- reduce-side products; every token contraction pairs kmap-permuted
  //      LDS rows or the P^T accumulator fragments
  {
    // (a) -M = -(Kt W), the state kernel's A operand (fragment order, prefill.h).
    //     Computed transposed, M^T = W^T Kt^T: rows d_in from sWt, columns d_out from Kt.
    T *nm_out = static_cast<T *>(a.NM) + blk * ((size_t)DK * DK);
#pragma unroll
    for (int nn = 0; nn < KPW; ++nn) {
      const int n = wave * KPW + nn;
      Frag<T> bk[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) bk[kb] = frag_sw<L::LDT>(sKt, 16 * n + col, kb * 32 + 8 * grp);
#pragma unroll
      for (int m2 = 0; m2 < KT; m2 += 2) {
        f32x4 acc[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          acc[h] = zero4();
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
            acc[h] = mma(acc[h], frag_sw<L::LDT>(sWt, 16 * (m2 + h) + col, kb * 32 + 8 * grp), bk[kb]);
        }
        // lane: column d_out, rows d_in = 16m + 4grp + e = 32(m >> 1) + kmap(grp, 4(m & 1) + e)
        // -> slots 4(m & 1) + e of operand block (t = n, kb = m >> 1): m = m2, m2 + 1 fill
        // the lane's 8 slots, one 16-byte store
        store8(nm_out + ((size_t)(n * (DK / 32) + (m2 >> 1)) * 64 + lane) * 8, -acc[0], -acc[1]);
      }
    }
    // (b) B = Kt U~, the state kernel's accumulator init (lane-major, prefill.h):
    //     lane col of state tile n feeds U~ row dv_of(n, col), so the product
    //     lands in the state's column order
    T *b_out = static_cast<T *>(a.Bc) + blk * ((size_t)DV * DK);
    Frag<T> ak[KPW][2];
#pragma unroll
    for (int mm = 0; mm < KPW; ++mm)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) ak[mm][kb] = frag_sw<L::LDT>(sKt, 16 * (wave * KPW + mm) + col, kb * 32 + 8 * grp);
#pragma unroll
    for (int n = 0; n < VT; ++n) {
      Frag<T> bu[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) bu[kb] = frag_sw<L::LDT>(sUt, dv_of(n, col), kb * 32 + 8 * grp);
      f32x4 acc[KPW];
#pragma unroll
      for (int mm = 0; mm < KPW; ++mm) {
        acc[mm] = zero4();
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) acc[mm] = mma(acc[mm], ak[mm][kb], bu[kb]);
      }
      // this wave's KPW row tiles m are consecutive: pairs share one 16-byte store
      T *bl = b_out + ((size_t)n * 64 + lane) * (4 * KT) + 4 * (wave * KPW);
      if constexpr (KPW % 2 == 0) {
#pragma unroll
        for (int mm = 0; mm < KPW; mm += 2) store8(bl + 4 * mm, acc[mm], acc[mm + 1]);
      } else {
#pragma unroll
        for (int mm = 0; mm < KPW; ++mm) store4(bl + 4 * mm, acc[mm]);
      }
    }
    // (c) Q' = Q e^gamma - P W and (d) O_loc = P U~, the output kernel's B
    //     operand and accumulator init (fragment order, token tile nt = wave),
    //     computed transposed with this wave's P^T fragments.  P is causal:
    //     k-blocks kb <= wave/2 only.
    const Frag<T> pb[2] = {frag_from_acc<T>(accP[0], accP[1]), frag_from_acc<T>(accP[2], accP[3])};
    const int nkb = (wave >> 1) + 1;
    const int r = rq;
    T *qp_out = static_cast<T *>(a.Qp) + blk * ((size_t)kChunk * DK) + (size_t)wave * (DK / 32) * 64 * 8;
#pragma unroll
    for (int m2 = 0; m2 < KT; m2 += 2) {
      f32x4 res[2];
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int m = m2 + h;
        const int d = 16 * m + 4 * grp;
        f32x4 qe = qacc[m] * qscale;
        const f32x4 gq = KDA ? *reinterpret_cast<const f32x4 *>(sGam + gam_at<DK>(r, d)) : zero4();
        f32x4 acc = zero4();
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          if (kb < nkb) acc = mma(acc, frag_sw<L::LDT>(sWt, 16 * m + col, kb * 32 + 8 * grp), pb[kb]);
#pragma unroll
        for (int e = 0; e < 4; ++e) qe[e] *= KDA ? __expf(gq[e]) : __expf((float)sGd[r]);
        res[h] = qe - acc;
      }
      // slots 4(m & 1) + e of block kb = m >> 1: m2 and m2 + 1 fill them, one 16-byte store
      store8(qp_out + ((size_t)(m2 >> 1) * 64 + lane) * 8, res[0], res[1]);
    }
    // O_loc^T rows of state tile m: lane col feeds U~ row dv_of(m, col)
    T *ol_out = static_cast<T *>(a.Ol) + blk * ((size_t)kChunk * DV);
#pragma unroll
    for (int m = 0; m < VT; ++m) {
      f32x4 acc = zero4();
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
        if (kb < nkb) acc = mma(acc, frag_sw<L::LDT>(sUt, dv_of(m, col), kb * 32 + 8 * grp), pb[kb]);
      store4(ol_out + ((size_t)m * 64 + lane) * 16 + 4 * wave, acc);
    }
  }
  if constexpr (OVL != 0) {
    // Every wave's factor stores have completed, so they sit in this XCD's
    // L2, before the block's ready flag is set there (an atomic: it executes
    // in the L2, where the walks' atomic reads of the flag see it).
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) __hip_atomic_fetch_or(a.ovl + kOvlFlags + blk, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (walker) {
      __syncthreads();  // the walk's exchange buffer reuses this item's LDS
      ovl_walk<T, DK, DV, KDA, OVL == 1>(a);
    }
  }
}

// The kernel's dynamic LDS exceeds the default 64 KiB limit for some
// instances: raise it once per device.
template <typename T, int DK, int DV, bool KDA, bool PRE, int OVL = 0>
static hipError_t set_lds_limit() {
  using L = LocalLayout<T, DK, DV, KDA>;
  constexpr int kMaxDevices = 64;
  static std::atomic<bool> done[kMaxDevices];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < kMaxDevices && done[dev].load(std::memory_order_relaxed)) return hipSuccess;
  const void *kern = reinterpret_cast<const void *>(&chunk_local_kernel<T, DK, DV, KDA, PRE, OVL>);
  if ((e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)L::bytes)) != hipSuccess)
    return e;
  if (dev < kMaxDevices) done[dev].store(true, std::memory_order_relaxed);
  return hipSuccess;
}

template <typename T, int DK, int DV, bool KDA, bool PRE>
static hipError_t launch_local_t(const PrefillArgs &a, hipStream_t stream) {
  using L = LocalLayout<T, DK, DV, KDA>;
  hipError_t e = set_lds_limit<T, DK, DV, KDA, PRE>();
  if (e != hipSuccess) return e;
  // one workgroup per (chunk, value head) block, padded to whole rounds of 8 q/k groups
  const long groups = (long)a.max_chunks * a.Hqk;
  const long items = (groups + 7) / 8 * 8 * (a.Hv / a.Hqk);
  hipLaunchKernelGGL((chunk_local_kernel<T, DK, DV, KDA, PRE>), dim3((unsigned)items), dim3(kLocalThreads), L::bytes,
                     stream, a);
  return hipGetLastError();
}

template <typename T, bool KDA, bool PRE>
static hipError_t dispatch_dims(const PrefillArgs &a, hipStream_t s) {
  if (a.Dk == 64 && a.Dv == 64) return launch_local_t<T, 64, 64, KDA, PRE>(a, s);
  if (a.Dk == 64 && a.Dv == 128) return launch_local_t<T, 64, 128, KDA, PRE>(a, s);
  if (a.Dk == 128 && a.Dv == 64) return launch_local_t<T, 128, 64, KDA, PRE>(a, s);
  return launch_local_t<T, 128, 128, KDA, PRE>(a, s);
}

template <typename T, bool KDA>
static hipError_t dispatch_pre(const PrefillArgs &a, hipStream_t s) {
  return a.pre ? dispatch_dims<T, KDA, true>(a, s) : dispatch_dims<T, KDA, false>(a, s);
}

hipError_t launch_chunk_local(const PrefillArgs &a, bool bf16, bool kda, hipStream_t s) {
  if (a.max_chunks == 0) return hipSuccess;
  if (bf16) return kda ? dispatch_pre<bf16_t, true>(a, s) : dispatch_pre<bf16_t, false>(a, s);
  return kda ? dispatch_pre<float, true>(a, s) : dispatch_pre<float, false>(a, s);
}

// ------------------------------------------------------------ overlapped launch
// One grid runs the chunk-local items and the whole-chain walks at once: the
// walk of chunk c starts as soon as chunk c's factors exist instead of after
// the last chunk-local block.  Walk workgroups come first in the grid, so
// they are resident (each waits on its first chunk) before the chunk-local
// workgroups fill the remaining slots; the chunk-local workgroups never wait,
// so the launch always drains.  Both roles pick their work from queues of the
// XCD they run on (xcc_id): the blocks of a head and its walks then share one
// L2, through which the factors and the ready flags pass.  Every XCD gets
// kOvlSlack workgroups of each role more than its share, so that a dispatch
// that deals the grid a little unevenly over the XCDs still covers every
// queue.
constexpr int kOvlSlack = 2;

__global__ __launch_bounds__(256) void overlap_setup_kernel(PrefillArgs a) {
  const long n = kOvlFlags + (long)a.max_chunks * a.Hv;
  for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n; i += (long)gridDim.x * 256) a.ovl[i] = 0;
  if (a.single && blockIdx.x == 0 && threadIdx.x == 0) a.status[0] = single_ok(a) ? 0 : kDevBadSeqlens;
}

hipError_t launch_overlap_setup(const PrefillArgs &a, hipStream_t stream) {
  const long n = kOvlFlags + (long)a.max_chunks * a.Hv;
  const long blocks = std::min<long>(256, (n + 255) / 256);
  hipLaunchKernelGGL(overlap_setup_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a);
  return hipGetLastError();
}

template <bool KDA, bool PRE, int OVL>
static hipError_t launch_ovl_t(PrefillArgs a, hipStream_t stream) {
  constexpr int DK = 128, DV = 128;
  using L = LocalLayout<bf16_t, DK, DV, KDA>;
  hipError_t e = set_lds_limit<bf16_t, DK, DV, KDA, PRE, OVL>();
  if (e != hipSuccess) return e;
  const long hx = ovl_heads(a.Hv, 0);  // the most heads any XCD serves
  const long walks = kXcdCount * ((long)a.N * hx * (DV / 16) + kOvlSlack);
  const long items = kXcdCount * ((long)a.max_chunks * hx + kOvlSlack);
  a.ovl_walk_wgs = (int)walks;
  hipLaunchKernelGGL((chunk_local_kernel<bf16_t, DK, DV, KDA, PRE, OVL>), dim3((unsigned)(walks + items)),
                     dim3(kLocalThreads), L::bytes, stream, a);
  return hipGetLastError();
}

hipError_t launch_overlapped(const PrefillArgs &a, hipStream_t s) {
  if (a.single) return a.pre ? launch_ovl_t<false, true, 1>(a, s) : launch_ovl_t<false, false, 1>(a, s);
  return a.pre ? launch_ovl_t<false, true, 2>(a, s) : launch_ovl_t<false, false, 2>(a, s);
}

}  // namespace hagdn
