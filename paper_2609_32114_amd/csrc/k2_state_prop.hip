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
// directly the B operand of Kt U: no LDS round trip, no lane shuffles.  W and
// Kt arrive kmap-permuted from the chunk-local kernel, one 16-byte load per
// fragment.
//
// Latency: the operands of chunk c+1 (W, Kt, U~, decay) do not depend on the
// state, so they are loaded into a second register set while chunk c is
// computed (bf16; the loop is unrolled by two so the sets swap roles without
// copies).  The chain then waits on memory only when a load takes longer than
// one chunk step.
//
// Workgroup -> (pair, tile) mapping is XCD-aware: consecutive workgroup ids
// are dealt round-robin to the 8 XCDs, so ids b, b+8, b+16, ... share an XCD;
// all d_v tiles of one (sequence, head) pair get ids in one such class and
// share that XCD's L2 for W and Kt, which every tile of the pair reads.
#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kXcds = 8;

// Four consecutive elements as loaded (bf16 bits, or fp32), converted at use.
__device__ __forceinline__ uint2 load_raw4(const bf16_t *p) { return *reinterpret_cast<const uint2 *>(p); }
__device__ __forceinline__ f32x4 load_raw4(const float *p) { return *reinterpret_cast<const f32x4 *>(p); }
__device__ __forceinline__ f32x4 raw4_to_f32(uint2 u) {
  f32x4 r;
  r[0] = __uint_as_float(u.x << 16);
  r[1] = __uint_as_float(u.x & 0xffff0000u);
  r[2] = __uint_as_float(u.y << 16);
  r[3] = __uint_as_float(u.y & 0xffff0000u);
  return r;
}
__device__ __forceinline__ f32x4 raw4_to_f32(f32x4 v) { return v; }

template <typename T> struct Raw4;
template <> struct Raw4<bf16_t> { using type = uint2; };
template <> struct Raw4<float> { using type = f32x4; };

// Everything one chunk step reads from memory, for one lane.
template <typename T, int DK, bool KDA>
struct ChunkOps {
  Frag<T> w[4][DK / 32];          // W rows 16m + col, d_k block kb
  Frag<T> kt[DK / 16][2];         // Kt rows 16t + col, token block kb
  typename Raw4<T>::type ut[4];   // U~^T[dv][16m + 4grp .. +3]
  f32x4 dec[KDA ? DK / 16 : 1];   // decay of rows 16t + 4grp .. +3 (GDN: [0][0])
};

template <typename T, int DK, int DV, bool KDA>
__device__ __forceinline__ void load_ops(ChunkOps<T, DK, KDA> &op, const T *__restrict__ Wg,
                                         const T *__restrict__ Ktg, const T *__restrict__ Utg,
                                         const float *__restrict__ decg, size_t blk, int dv,
                                         int col, int grp) {
  const T *w = Wg + blk * ((size_t)kChunk * DK);
  const T *kt = Ktg + blk * ((size_t)DK * kChunk);
  const T *ut = Utg + blk * ((size_t)DV * kChunk) + (size_t)dv * kChunk;
  const float *dec = decg + blk * DK;
#pragma unroll
  for (int m = 0; m < 4; ++m)
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) op.w[m][kb] = load_frag(w + (16 * m + col) * DK + kb * 32, grp);
#pragma unroll
  for (int t = 0; t < DK / 16; ++t)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) op.kt[t][kb] = load_frag(kt + (16 * t + col) * kChunk + kb * 32, grp);
#pragma unroll
  for (int m = 0; m < 4; ++m) op.ut[m] = load_raw4(ut + 16 * m + 4 * grp);
  if constexpr (KDA) {
#pragma unroll
    for (int t = 0; t < DK / 16; ++t) op.dec[t] = load4(dec + 16 * t + 4 * grp);
  } else {
    op.dec[0][0] = dec[0];
  }
}

// One chunk step on the state tile H (rows 16t + 4grp + e, column dv).
template <typename T, int DK, int DV, bool KDA>
__device__ __forceinline__ void chunk_step(f32x4 (&H)[DK / 16], const ChunkOps<T, DK, KDA> &op,
                                           T *__restrict__ Ug, T *__restrict__ Hsg, size_t blk,
                                           int dv, int grp) {
  constexpr int KT = DK / 16;
  // 5-read: S_c as MFMA fragments; the same fragments are the snapshot for
  // operator #6, stored [d_v][d_k] kmap-permuted along d_k (16-byte stores)
  Frag<T> hb[DK / 32];
#pragma unroll
  for (int kb = 0; kb < DK / 32; ++kb) hb[kb] = frag_from_acc<T>(H[2 * kb], H[2 * kb + 1]);
  T *hs = Hsg + blk * ((size_t)DV * DK) + (size_t)dv * DK;
#pragma unroll
  for (int kb = 0; kb < DK / 32; ++kb) store_frag(hs + kb * 32, hb[kb], grp);
  // U = U~ + (-W) S_c^T   (rows = tokens, columns = this tile's d_v; W is stored negated)
  f32x4 U[4];
#pragma unroll
  for (int m = 0; m < 4; ++m) {
    U[m] = raw4_to_f32(op.ut[m]);
#pragma unroll
    for (int kb = 0; kb < DK / 32; ++kb) U[m] = mma(U[m], op.w[m][kb], hb[kb]);
  }
  // U in the operand precision, as MFMA fragments: used below and stored for
  // operator #6 ([d_v][token], kmap-permuted along tokens)
  Frag<T> ub[2];
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) ub[kb] = frag_from_acc<T>(U[2 * kb], U[2 * kb + 1]);
  T *uo = Ug + blk * ((size_t)DV * kChunk) + (size_t)dv * kChunk;
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) store_frag(uo + kb * 32, ub[kb], grp);
  // 5-update: S^T <- Diag(e^gamma_last) S^T + Kt U
  if constexpr (KDA) {
#pragma unroll
    for (int t = 0; t < KT; ++t) H[t] *= op.dec[t];
  } else {
    const float d0 = op.dec[0][0];
#pragma unroll
    for (int t = 0; t < KT; ++t) H[t] *= d0;
  }
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) H[t] = mma(H[t], op.kt[t][kb], ub[kb]);
}

// ---------------------------------------------------------------------------
// bf16: pipelined variant.  Workgroup = 1 chain wave + kLoaderWaves loader
// waves.  The loaders stream each chunk's operands (W, Kt, this tile's 16
// columns of U~, the decay) as 16-byte pieces dealt round-robin over their
// lanes; every lane keeps D chunks of pieces in flight in registers and writes
// one chunk per step into a double-buffered LDS stage (rows padded by 16 B so
// the chain wave's 16-byte fragment reads spread over the banks).  The chain
// wave reads the stage and runs chunk_step.  One barrier per chunk: the stage
// the chain reads in step c was written in step c-1, and the stage written in
// step c was last read in step c-1.  A piece loaded in step c is consumed in
// step c+D, so D chunk steps of memory latency are covered.
constexpr int kLoaderWaves = 7;
constexpr int kPipeDepth = 8;

template <int DK>
struct Stage {
  static constexpr int LDW = DK * 2 + 16;        // bytes per W row (64 rows)
  static constexpr int LDKT = kChunk * 2 + 16;   // bytes per Kt row (DK rows)
  static constexpr int LDUT = kChunk * 2 + 16;   // bytes per U~ row (16 rows)
  static constexpr int off_w = 0;
  static constexpr int off_kt = off_w + kChunk * LDW;
  static constexpr int off_ut = off_kt + DK * LDKT;
  static constexpr int off_dec = off_ut + 16 * LDUT;
  static constexpr int bytes = off_dec + DK * 4;
  // 16-byte pieces of one chunk: W, Kt, U~ tile, decay (KDA: DK floats, GDN: one piece)
  static constexpr int nW = kChunk * DK / 8, nKt = DK * kChunk / 8, nUt = 16 * kChunk / 8;
  template <bool KDA> static constexpr int pieces() { return nW + nKt + nUt + (KDA ? DK / 4 : 1); }
  template <bool KDA> static constexpr int slots() {
    return (pieces<KDA>() + 64 * kLoaderWaves - 1) / (64 * kLoaderWaves);
  }
};

template <int DK, int DV, bool KDA, int D>
__global__ __launch_bounds__(64 * (1 + kLoaderWaves)) void state_prop_pipe_kernel(PrefillArgs a) {
  using S = Stage<DK>;
  using T = bf16_t;
  constexpr int NT = DV / 16;
  constexpr int KT = DK / 16;
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / NT) * kXcds + xcd;
  const int tile = slot % NT;
  if (pair >= a.N * a.Hv) return;  // uniform for the workgroup
  const int n = pair / a.Hv, h = pair % a.Hv;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int dv = tile * 16 + col;
  const int4 si = a.seq_info[n];
  const int nch = si.y;
  extern __shared__ __align__(16) unsigned char smem[];
  // Both wave roles run npad = nch rounded up to D steps (one barrier each);
  // steps past nch do no chain work.  Every loader load is unconditional (chunk
  // index clamped, dead slots reload a live piece), so the number of loads in
  // flight is the same on every path and each LDS write waits only for its own
  // chunk's loads.
  const int npad = (nch + D - 1) / D * D;

  if (wave == 0) {
    // ------------------------------------------------------------ chain wave
    f32x4 H[KT];
    const size_t sbase = ((size_t)n * a.Hv + h) * DK * DV;
#pragma unroll
    for (int t = 0; t < KT; ++t)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        H[t][e] = a.s0 ? a.s0[sbase + (size_t)(16 * t + 4 * grp + e) * DV + dv] : 0.f;
    T *__restrict__ Ug = static_cast<T *>(a.U);
    T *__restrict__ Hsg = static_cast<T *>(a.Hs);
    if (nch > 0) __syncthreads();  // prologue: stage 0 holds chunk 0
    for (int c = 0; c < npad; ++c) {
      if (c >= nch) {
        __syncthreads();
        continue;
      }
      const unsigned char *sb = smem + (c & 1) * S::bytes;
      ChunkOps<T, DK, KDA> op;
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb)
          op.w[m][kb] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const uint4 *>(sb + S::off_w + (16 * m + col) * S::LDW +
                                                       (kb * 32 + 8 * grp) * 2));
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          op.kt[t][kb] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const uint4 *>(sb + S::off_kt + (16 * t + col) * S::LDKT +
                                                       (kb * 32 + 8 * grp) * 2));
#pragma unroll
      for (int m = 0; m < 4; ++m)
        op.ut[m] = *reinterpret_cast<const uint2 *>(sb + S::off_ut + col * S::LDUT + (16 * m + 4 * grp) * 2);
      const float *sdec = reinterpret_cast<const float *>(sb + S::off_dec);
      if constexpr (KDA) {
#pragma unroll
        for (int t = 0; t < KT; ++t) op.dec[t] = *reinterpret_cast<const f32x4 *>(sdec + 16 * t + 4 * grp);
      } else {
        op.dec[0][0] = sdec[0];
      }
      chunk_step<T, DK, DV, KDA>(H, op, Ug, Hsg, (size_t)(si.x + c) * a.Hv + h, dv, grp);
      __syncthreads();
    }
    if (a.s_final) {
#pragma unroll
      for (int t = 0; t < KT; ++t)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          a.s_final[sbase + (size_t)(16 * t + 4 * grp + e) * DV + dv] = H[t][e];
    }
  } else {
    // ----------------------------------------------------------- loader waves
    constexpr int NS = S::template slots<KDA>();
    constexpr int NP = S::template pieces<KDA>();
    // per slot: byte address of the piece in chunk block 0 of this head, byte
    // stride between consecutive (chunk, head) blocks, LDS byte offset
    const unsigned char *src0[NS];
    size_t bstride[NS];
    int loff[NS];
    bool live[NS];
#pragma unroll
    for (int i = 0; i < NS; ++i) {
      const int q = i * 64 * kLoaderWaves + (wave - 1) * 64 + lane;
      live[i] = q < NP;
      const unsigned char *base;
      size_t goff, stride;
      int lo;
      if (q < S::nW) {
        const int row = q / (DK / 8), pc = q % (DK / 8);
        base = static_cast<const unsigned char *>(a.W);
        stride = (size_t)kChunk * DK * 2;
        goff = (size_t)(row * DK + pc * 8) * 2;
        lo = S::off_w + row * S::LDW + pc * 16;
      } else if (q < S::nW + S::nKt) {
        const int r = q - S::nW, row = r / 8, pc = r % 8;
        base = static_cast<const unsigned char *>(a.Kt);
        stride = (size_t)DK * kChunk * 2;
        goff = (size_t)(row * kChunk + pc * 8) * 2;
        lo = S::off_kt + row * S::LDKT + pc * 16;
      } else if (q < S::nW + S::nKt + S::nUt) {
        const int r = q - S::nW - S::nKt, row = r / 8, pc = r % 8;
        base = static_cast<const unsigned char *>(a.Ut);
        stride = (size_t)DV * kChunk * 2;
        goff = (size_t)((tile * 16 + row) * kChunk + pc * 8) * 2;
        lo = S::off_ut + row * S::LDUT + pc * 16;
      } else if (live[i]) {
        const int r = q - S::nW - S::nKt - S::nUt;
        base = reinterpret_cast<const unsigned char *>(a.dec);
        stride = (size_t)DK * 4;
        goff = (size_t)r * 16;
        lo = S::off_dec + r * 16;
      } else {  // dead slot: reloads the first W piece, never written to LDS
        base = static_cast<const unsigned char *>(a.W);
        stride = (size_t)kChunk * DK * 2;
        goff = 0;
        lo = 0;
      }
      src0[i] = base + (size_t)h * stride + goff;  // block of chunk 0 = si.x * Hv + h
      bstride[i] = stride;
      loff[i] = lo;
    }
    const size_t head_blocks = (size_t)a.Hv;  // blocks between consecutive chunks of a head
    u32x4 R[D][NS];
    auto issue = [&](u32x4 (&r)[NS], int c) {
      const size_t blk = (size_t)(si.x + min(c, nch - 1)) * head_blocks;
#pragma unroll
      for (int i = 0; i < NS; ++i) r[i] = *reinterpret_cast<const u32x4 *>(src0[i] + blk * bstride[i]);
    };
    auto write = [&](const u32x4 (&r)[NS], int c) {
      unsigned char *sb = smem + (c & 1) * S::bytes;
#pragma unroll
      for (int i = 0; i < NS; ++i)
        if (live[i]) *reinterpret_cast<u32x4 *>(sb + loff[i]) = r[i];
    };
    if (nch > 0) {
      // prologue: chunks 0..D-1 in flight, chunk 0 into stage 0, refill set 0 with chunk D
#pragma unroll
      for (int u = 0; u < D; ++u) issue(R[u], u);
      write(R[0], 0);
      issue(R[0], D);
      __syncthreads();
      for (int c0 = 0; c0 < npad; c0 += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
          // chunk c+1 (loaded D steps ago) into the stage the chain reads next;
          // past the end this rewrites the last chunk into a stage nobody reads
          write(R[(u + 1) % D], c0 + u + 1);
          issue(R[(u + 1) % D], c0 + u + 1 + D);
          __syncthreads();
        }
      }
    }
  }
}

template <typename T, int DK, int DV, bool KDA>
__global__ __launch_bounds__(64) void state_prop_kernel(PrefillArgs a) {
  constexpr int NT = DV / 16;   // d_v tiles per head
  constexpr int KT = DK / 16;   // accumulator tiles of the state (d_k rows)
  constexpr bool kPrefetch = sizeof(T) == 2;  // fp32 operands would not fit twice
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / NT) * kXcds + xcd;
  const int tile = slot % NT;
  if (pair >= a.N * a.Hv) return;
  const int n = pair / a.Hv, h = pair % a.Hv;
  const int lane = threadIdx.x, col = lane & 15, grp = lane >> 4;
  const int dv = tile * 16 + col;  // state column this lane holds
  const int4 si = a.seq_info[n];   // {first chunk, chunks, start, length}
  const int nch = si.y;

  // state tile: H[t][e] = S^T[16t + 4grp + e][dv]
  f32x4 H[KT];
  const size_t sbase = ((size_t)n * a.Hv + h) * DK * DV;
#pragma unroll
  for (int t = 0; t < KT; ++t)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      H[t][e] = a.s0 ? a.s0[sbase + (size_t)(16 * t + 4 * grp + e) * DV + dv] : 0.f;

  const T *__restrict__ Wg = static_cast<const T *>(a.W);
  const T *__restrict__ Utg = static_cast<const T *>(a.Ut);
  const T *__restrict__ Ktg = static_cast<const T *>(a.Kt);
  T *__restrict__ Ug = static_cast<T *>(a.U);
  T *__restrict__ Hsg = static_cast<T *>(a.Hs);
  const float *__restrict__ decg = a.dec;
  auto blk_of = [&](int c) { return (size_t)(si.x + c) * a.Hv + h; };

  if constexpr (kPrefetch) {
    ChunkOps<T, DK, KDA> A, B;
    if (nch > 0) load_ops<T, DK, DV, KDA>(A, Wg, Ktg, Utg, decg, blk_of(0), dv, col, grp);
    for (int c = 0; c < nch; c += 2) {
      // operands of chunk c+1 (clamped: the last step reloads its own chunk)
      load_ops<T, DK, DV, KDA>(B, Wg, Ktg, Utg, decg, blk_of(min(c + 1, nch - 1)), dv, col, grp);
      chunk_step<T, DK, DV, KDA>(H, A, Ug, Hsg, blk_of(c), dv, grp);
      if (c + 1 < nch) {
        load_ops<T, DK, DV, KDA>(A, Wg, Ktg, Utg, decg, blk_of(min(c + 2, nch - 1)), dv, col, grp);
        chunk_step<T, DK, DV, KDA>(H, B, Ug, Hsg, blk_of(c + 1), dv, grp);
      }
    }
  } else {
    for (int c = 0; c < nch; ++c) {
      ChunkOps<T, DK, KDA> A;
      load_ops<T, DK, DV, KDA>(A, Wg, Ktg, Utg, decg, blk_of(c), dv, col, grp);
      chunk_step<T, DK, DV, KDA>(H, A, Ug, Hsg, blk_of(c), dv, grp);
    }
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
  if constexpr (sizeof(T) == 2) {
    constexpr int lds = 2 * Stage<DK>::bytes;
    static bool attr_set = false;
    if (!attr_set) {
      hipError_t e = hipFuncSetAttribute(
          reinterpret_cast<const void *>(&state_prop_pipe_kernel<DK, DV, KDA, kPipeDepth>),
          hipFuncAttributeMaxDynamicSharedMemorySize, lds);
      if (e != hipSuccess) return e;
      attr_set = true;
    }
    hipLaunchKernelGGL((state_prop_pipe_kernel<DK, DV, KDA, kPipeDepth>), dim3((unsigned)blocks),
                       dim3(64 * (1 + kLoaderWaves)), lds, stream, a);
  } else {
    hipLaunchKernelGGL((state_prop_kernel<T, DK, DV, KDA>), dim3((unsigned)blocks), dim3(64), 0,
                       stream, a);
  }
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
