// k3_segments.hip -- the Reduce phase of chunkwise delta-rule prefill
// (paper Sec. 2.1, operator #5 H) fused with the final Map (operator #6 O),
// parallelised over segments of the chunk chain (paper Sec. 4, the
// Chunk-Seg-Seg mapping).  Used when chains are long enough for the segment
// maps to pay; k2_state_prop.hip walks short chains whole.
//
// Per chunk the chunk-local kernel has reduced operator #5 to an affine map of
// the state entering the chunk (S^T, d_k x d_v):
//     S^T_{c+1} = D S^T_c + NM S^T_c + B,     NM = -Kt W,  B = Kt U~,  D = Diag(e^gamma_last)
// so the critical path of one chunk step is a single d_k x d_k by d_k x d_v
// product.  Affine maps compose: over a segment of chunks they give one map
// S^T_out = A S^T_in + B_seg.  Two kernels:
//
//   seg_transfer  one workgroup per (segment, value head, part): runs the
//                 segment's chunk chain on A (part 0, from I, no B term) or on
//                 B_seg (part 1, from 0) and stores the segment map -- only for
//                 segments that another segment of the same sequence follows
//                 (fp32; the bf16 maps run on the staged walk, seg_map_kernel
//                 in k2_walk.hip);
//   seg_state     one workgroup per (segment, value head): applies the maps of
//                 the earlier segments of its sequence (a short chain of
//                 d_k x d_k products; the first segment's B_seg already
//                 carries the initial state), then walks its own chunks,
//                 updating the state and emitting o; the last segment of a
//                 sequence writes the final state.
// The serial depth drops from the number of chunks n to about
// seg_chunks (transfer) + n / seg_chunks (prefix) + seg_chunks (walk).
//
// Head-resident workgroups (paper Sec. 4, head-level mapping): one workgroup
// keeps a whole d_k x (columns) state on one CU.  Its four waves split the
// columns -- wave w owns columns [w NCOL/4, (w+1) NCOL/4) of every row, as
// NCOL/64 column tiles x d_k/16 row tiles of fp32 MFMA accumulators -- so the
// columns evolve independently (paper Sec. 4, "Computation Splitting") and
// each wave turns its own accumulators into the B operand of the next product
// (device.h: an accumulator pair IS a B fragment under the kmap slot order):
// no cross-wave exchange of the state, no reduction.  What the waves share
// are the chunk's NM (and Q') blocks: staged once per step into LDS, in the
// fragment order they are stored in, and read by every wave as contiguous
// 16-byte fragments.  One copy per (segment, head) instead of one per column
// tile keeps L2 traffic at the compulsory bytes.
//
// Chunk-first order (paper Sec. 5, "Cross-Chunk"): S_c is read by everything
// that needs it -- including operator #6,
//     O^T = S_c Q'^T + O_loc^T        (factors from the chunk-local kernel)
// -- before it is overwritten; the output products reuse the B fragments of
// S_c as A operands and run off the state's critical path.
//
// Pipeline: chunk c's NM/Q' are fetched into a register ring three steps
// ahead and written to LDS stage c % NSTAGE at the end of the step before; the
// per-lane B, O_loc and decay of chunk c are fetched two steps ahead into a
// register ring.  Fetches
// are unconditional (chunk index clamped) so every path keeps the same number
// of memory operations in flight.
//
// Workgroup -> work mapping is XCD-aware: consecutive workgroup ids are dealt
// round-robin to the 8 XCDs; ids b, b+8, ... share an XCD and its L2.
#include <type_traits>

#include "device.h"
#include "prefill.h"

namespace hagdn {

constexpr int kXcds = 8;
constexpr int kHeadThreads = 256;  // four waves per head-resident workgroup

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

// Range-checked stores: a buffer resource over [base, base + bytes); lanes whose
// byte offset falls outside (negative offsets included) store nothing.  Stores
// that need no branch keep the compiler's memory-counter waits exact.
constexpr int kBufferWord3 = 0x00020000;  // gfx9 buffer resource word 3 (raw, 32-bit format)
__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_over(void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)bytes, kBufferWord3);
}
__device__ __forceinline__ void store4_checked(__amdgpu_buffer_rsrc_t r, int byte_off, bf16_t, f32x4 v) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  u32x2 u;
  u[0] = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  u[1] = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  __builtin_amdgcn_raw_buffer_store_b64(u, r, byte_off, 0, 0);
}
__device__ __forceinline__ void store4_checked(__amdgpu_buffer_rsrc_t r, int byte_off, float, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, byte_off, 0, 0);
}
// Eight consecutive elements (lo then hi).
__device__ __forceinline__ void store8_checked(__amdgpu_buffer_rsrc_t r, int byte_off, bf16_t, f32x4 lo, f32x4 hi) {
  u32x4 u;
  u[0] = (uint32_t)f32_to_bf16(lo[0]) | ((uint32_t)f32_to_bf16(lo[1]) << 16);
  u[1] = (uint32_t)f32_to_bf16(lo[2]) | ((uint32_t)f32_to_bf16(lo[3]) << 16);
  u[2] = (uint32_t)f32_to_bf16(hi[0]) | ((uint32_t)f32_to_bf16(hi[1]) << 16);
  u[3] = (uint32_t)f32_to_bf16(hi[2]) | ((uint32_t)f32_to_bf16(hi[3]) << 16);
  __builtin_amdgcn_raw_buffer_store_b128(u, r, byte_off, 0, 0);
}
__device__ __forceinline__ void store8_checked(__amdgpu_buffer_rsrc_t r, int byte_off, float, f32x4 lo, f32x4 hi) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, lo), r, byte_off, 0, 0);
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, hi), r, byte_off + 16, 0, 0);
}

// Workgroup id -> work index: items of per_item workgroups each are dealt
// round-robin to the XCDs, all workgroups of one item on one XCD.
__device__ __forceinline__ int xcd_item(int b, int per_item) {
  const int xcd = b % kXcds, slot = b / kXcds;
  return ((slot / per_item) * kXcds + xcd) * per_item + slot % per_item;
}

// f(integral_constant<i>) for i = LO .. HI-1, unrolled at compile time.
template <int LO, int HI, typename F>
__device__ __forceinline__ void static_for(F &&f) {
  if constexpr (LO < HI) {
    f(std::integral_constant<int, LO>{});
    static_for<LO + 1, HI>(f);
  }
}

// LDS stage of one chain step: the d_k x d_k operator block (NM or a segment's
// A) and, for output steps, the 64 x d_k Q' block; both in fragment order.
template <typename T, int DK, bool WITH_QP>
struct Stage {
  static constexpr int NM_BYTES = DK * DK * (int)sizeof(T);
  static constexpr int QP_BYTES = WITH_QP ? kChunk * DK * (int)sizeof(T) : 0;
  static constexpr int BYTES = NM_BYTES + QP_BYTES;
  static constexpr int NM_V = NM_BYTES / (kHeadThreads * 16);  // 16-byte vectors per thread
  static constexpr int NV = BYTES / (kHeadThreads * 16);
  static constexpr int NSTAGE = 2 * BYTES <= 128 * 1024 ? 2 : 1;
  static_assert(NV * kHeadThreads * 16 == BYTES, "stage must split into 16-byte vectors");
};

// Thread tid's share of a stage: vector i is bytes [(i*256 + tid)*16, +16) of
// the NM block (i < NM_V) or of the Q' block.
template <int NM_V, int NV>
__device__ __forceinline__ void stage_fetch(u32x4 (&r)[NV], const char *nm, const char *qp, int tid) {
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const char *base = i < NM_V ? nm + i * 4096 : qp + (i - NM_V) * 4096;
    r[i] = *reinterpret_cast<const u32x4 *>(base + tid * 16);
  }
}
template <int NV>
__device__ __forceinline__ void stage_put(const u32x4 (&r)[NV], char *st, int tid) {
#pragma unroll
  for (int i = 0; i < NV; ++i) *reinterpret_cast<u32x4 *>(st + i * 4096 + tid * 16) = r[i];
}

// Fragment (block b of a fragment-order region in LDS) for this lane.
template <typename T>
__device__ __forceinline__ Frag<T> lds_frag(const char *region, int b, int lane) {
  const char *p = region + ((size_t)b * 64 + lane) * 8 * sizeof(T);
  if constexpr (sizeof(T) == 2) {
    return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(p));
  } else {
    const f32x4 x = *reinterpret_cast<const f32x4 *>(p), y = *reinterpret_cast<const f32x4 *>(p + 16);
    return __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7);
  }
}

// The columns of a d_k x NCOL state (or map) held by one wave.
template <typename T, int DK, int NCOL>
struct HeadState {
  static constexpr int CT = NCOL / 64;  // 16-column tiles per wave
  static constexpr int RT = DK / 16;    // 16-row tiles
  static constexpr int KB = DK / 32;    // 32-row k-blocks
  f32x4 H[CT][RT];       // H[ct][rt][e] = X[16rt + 4grp + e][col0 + 16ct + col]
  Frag<T> hb[CT][KB];    // X as B operand, k-block kb (kmap slot order)

  __device__ __forceinline__ void make_hb() {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) hb[ct][kb] = frag_from_acc<T>(H[ct][2 * kb], H[ct][2 * kb + 1]);
  }
  // H[ct][rt] += sum_kb M(rt, kb) hb[ct][kb], M in fragment order in LDS.
  // k-block outermost: the CT x RT accumulators are independent, so
  // consecutive products never wait on each other.  The LDS reads of k-block
  // kb+1 are issued before the products of kb, with scheduling fences in
  // between, so at most two k-blocks of fragments are held at once.
  // after(kb) runs behind the products of k-block kb (other work to overlap).
  template <typename After>
  __device__ __forceinline__ void mm_lds(const char *m, int lane, After &&after) {
    Frag<T> f[2][RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) f[0][rt] = lds_frag<T>(m, rt * KB, lane);
    static_for<0, KB>([&](auto kbc) {
      constexpr int kb = decltype(kbc)::value;
      if constexpr (kb + 1 < KB) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) f[(kb + 1) & 1][rt] = lds_frag<T>(m, rt * KB + kb + 1, lane);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int ct = 0; ct < CT; ++ct) H[ct][rt] = mma(H[ct][rt], f[kb & 1][rt], hb[ct][kb]);
      after(kbc);
      __builtin_amdgcn_sched_barrier(0);
    });
  }
  __device__ __forceinline__ void mm_lds(const char *m, int lane) {
    mm_lds(m, lane, [](auto) {});
  }
};

// Per-lane operands of one chunk step, fetched two steps ahead.
template <typename T, int DK, int NCOL, bool KDA, bool WITH_B, bool WITH_OUT>
struct LaneOps {
  static constexpr int CT = NCOL / 64, RT = DK / 16;
  typename Raw4<T>::type b[WITH_B ? CT : 1][RT];   // B block (tile, rt)
  typename Raw4<T>::type ol[WITH_OUT ? CT : 1][4]; // O_loc block (token tile, tile)
  f32x4 dec[KDA ? RT : 1];                         // decay of rows 16rt + 4grp + e (GDN: dec[0][0])
};

// n raw 4-element groups that lie contiguously at p (16-byte loads).
template <int N>
__device__ __forceinline__ void load_raw4_run(uint2 (&r)[N], const bf16_t *p) {
#pragma unroll
  for (int i = 0; i < N / 2; ++i) {
    const u32x4 v = *reinterpret_cast<const u32x4 *>(p + 8 * i);
    r[2 * i] = make_uint2(v[0], v[1]);
    r[2 * i + 1] = make_uint2(v[2], v[3]);
  }
}
template <int N>
__device__ __forceinline__ void load_raw4_run(f32x4 (&r)[N], const float *p) {
#pragma unroll
  for (int i = 0; i < N; ++i) r[i] = *reinterpret_cast<const f32x4 *>(p + 4 * i);
}

template <typename T, int DK, int NCOL, bool KDA, bool WITH_B, bool WITH_OUT>
__device__ __forceinline__ void lane_fetch(LaneOps<T, DK, NCOL, KDA, WITH_B, WITH_OUT> &op, const PrefillArgs &a,
                                           size_t blk, int w, int lane) {
  constexpr int CT = NCOL / 64, RT = DK / 16;
  const int t0 = w * CT;  // first column tile of this wave
  if constexpr (WITH_B) {
    // lane-major B (prefill.h): this lane's RT groups of tile t0 + ct are contiguous
    const T *bt = static_cast<const T *>(a.Bc) + blk * ((size_t)DK * a.Dv);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) load_raw4_run(op.b[ct], bt + ((size_t)(t0 + ct) * 64 + lane) * (4 * RT));
  }
  if constexpr (WITH_OUT) {
    const T *ol = static_cast<const T *>(a.Ol) + blk * ((size_t)kChunk * a.Dv);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct) load_raw4_run(op.ol[ct], ol + ((size_t)(t0 + ct) * 64 + lane) * 16);
  }
  if constexpr (KDA) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) op.dec[rt] = load4(a.dec + blk * DK + 16 * rt + 4 * (lane >> 4));
  } else {
    op.dec[0][0] = a.dec[blk * DK];
  }
}

// H <- D H (+ B): the state-independent part of a chunk step.
template <typename T, int DK, int NCOL, bool KDA, bool WITH_B, bool WITH_OUT>
__device__ __forceinline__ void chunk_init(HeadState<T, DK, NCOL> &hs,
                                           const LaneOps<T, DK, NCOL, KDA, WITH_B, WITH_OUT> &op) {
  constexpr int CT = NCOL / 64, RT = DK / 16;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const f32x4 d = KDA ? op.dec[KDA ? rt : 0]
                          : f32x4{op.dec[0][0], op.dec[0][0], op.dec[0][0], op.dec[0][0]};
      hs.H[ct][rt] = d * hs.H[ct][rt];
      if constexpr (WITH_B) hs.H[ct][rt] += raw4_to_f32(op.b[WITH_B ? ct : 0][rt]);
    }
}

// Walks chunks [0, nch) (nch >= 1) of blocks blk(c) from the state in hs: the
// pipeline described at the top of the file.  WITH_OUT emits operator #6
// through out(c, pend) one step late.
template <typename T, int DK, int NCOL, bool KDA, bool WITH_B, bool WITH_OUT, typename BlkFn, typename OutFn>
__device__ __forceinline__ void walk_chunks(HeadState<T, DK, NCOL> &hs, const PrefillArgs &a, int nch,
                                            BlkFn blk, OutFn out, char *lds) {
  using S = Stage<T, DK, WITH_OUT>;
  using Ops = LaneOps<T, DK, NCOL, KDA, WITH_B, WITH_OUT>;
  constexpr int CT = NCOL / 64;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const char *NMg = static_cast<const char *>(a.NM);
  const char *QPg = static_cast<const char *>(a.Qp);
  auto fetch_stage = [&](u32x4 (&r)[S::NV], int c) {
    const size_t b = blk(c);
    stage_fetch<S::NM_V>(r, NMg + b * S::NM_BYTES, WITH_OUT ? QPg + b * S::QP_BYTES : nullptr, tid);
  };
  auto stage_at = [&](int c) { return lds + (c % S::NSTAGE) * S::BYTES; };

  u32x4 sreg[2][S::NV];  // NM/Q' of chunk c: slot c & 1, fetched two steps ahead
  Ops ops[2];
  f32x4 pend[CT][4];
  fetch_stage(sreg[0], 0);
  fetch_stage(sreg[1], 1);
  lane_fetch(ops[0], a, blk(0), w, lane);
  lane_fetch(ops[1], a, blk(1), w, lane);
  if constexpr (S::NSTAGE == 1) __syncthreads();  // the caller may still read the stage memory
  stage_put(sreg[0], stage_at(0), tid);
  fetch_stage(sreg[0], 2);

  // Memory work of a step, as a sequence of items issued in NSL slices behind
  // the product groups so the address, LDS and matrix units overlap: the LDS
  // stage of chunk c+1 (vectors 0..NV-1), the stage registers of chunk c+3,
  // then this slot's per-lane operands of chunk c+2 (B, decay, O_loc last: the
  // output products read the O_loc being replaced first).
  constexpr int RT = DK / 16;
  constexpr int NB = WITH_B ? CT * (sizeof(T) == 2 ? RT / 2 : RT) : 0;  // 16-byte B loads
  constexpr int NO = WITH_OUT ? CT * (sizeof(T) == 2 ? 2 : 4) : 0;       // 16-byte O_loc loads
  constexpr int NI = 2 * S::NV + NB + 1 + NO;
  constexpr int NSL = WITH_OUT ? 2 * (DK / 32) : DK / 32;
  auto step = [&](auto slot_c, int c) {
    constexpr int u = decltype(slot_c)::value;  // c & 1
    __syncthreads();  // stage of chunk c complete; every wave is past step c-1
    if constexpr (WITH_OUT) out(c - 1, pend);  // chunk -1 stores nothing
    hs.make_hb();
    chunk_init(hs, ops[u]);
    const char *st = stage_at(c);
    char *st_next = stage_at(c + 1);
    const size_t bs = blk(c + 3), bl = blk(c + 2);
    const char *nm3 = NMg + bs * S::NM_BYTES;
    const char *qp3 = WITH_OUT ? QPg + bs * S::QP_BYTES : nullptr;
    const T *bt = static_cast<const T *>(a.Bc) + bl * ((size_t)DK * a.Dv) + ((size_t)w * CT * 64 + lane) * (4 * RT);
    const T *olp = static_cast<const T *>(a.Ol) + bl * ((size_t)kChunk * a.Dv) + ((size_t)w * CT * 64 + lane) * 16;
    auto item = [&](auto ic) {
      constexpr int i = decltype(ic)::value;
      if constexpr (i < S::NV) {
        *reinterpret_cast<u32x4 *>(st_next + i * 4096 + tid * 16) = sreg[u ^ 1][i];
      } else if constexpr (i < 2 * S::NV) {
        constexpr int j = i - S::NV;
        const char *base = j < S::NM_V ? nm3 + j * 4096 : qp3 + (j - S::NM_V) * 4096;
        sreg[u ^ 1][j] = *reinterpret_cast<const u32x4 *>(base + tid * 16);
      } else if constexpr (i < 2 * S::NV + NB) {
        constexpr int j = i - 2 * S::NV;
        if constexpr (sizeof(T) == 2) {
          constexpr int ct = j / (RT / 2), q = j % (RT / 2);
          const u32x4 v = *reinterpret_cast<const u32x4 *>(bt + (size_t)ct * 64 * 4 * RT + 8 * q);
          ops[u].b[ct][2 * q] = make_uint2(v[0], v[1]);
          ops[u].b[ct][2 * q + 1] = make_uint2(v[2], v[3]);
        } else {
          constexpr int ct = j / RT, rt = j % RT;
          ops[u].b[ct][rt] = *reinterpret_cast<const typename Raw4<T>::type *>(bt + (size_t)ct * 64 * 4 * RT + 4 * rt);
        }
      } else if constexpr (i == 2 * S::NV + NB) {
        if constexpr (KDA) {
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) ops[u].dec[rt] = load4(a.dec + bl * DK + 16 * rt + 4 * (lane >> 4));
        } else {
          ops[u].dec[0][0] = a.dec[bl * DK];
        }
      } else {
        constexpr int j = i - 2 * S::NV - NB - 1;
        if constexpr (sizeof(T) == 2) {
          constexpr int ct = j / 2, q = j % 2;
          const u32x4 v = *reinterpret_cast<const u32x4 *>(olp + (size_t)ct * 64 * 16 + 8 * q);
          ops[u].ol[ct][2 * q] = make_uint2(v[0], v[1]);
          ops[u].ol[ct][2 * q + 1] = make_uint2(v[2], v[3]);
        } else {
          constexpr int ct = j / 4, nt = j % 4;
          ops[u].ol[ct][nt] = *reinterpret_cast<const typename Raw4<T>::type *>(olp + (size_t)ct * 64 * 16 + 4 * nt);
        }
      }
    };
    // slice g issues items [g NI / NSL, (g+1) NI / NSL); with a single stage
    // every item waits until the stage's readers are done
    auto slice = [&](auto gc) {
      constexpr int g = decltype(gc)::value;
      if constexpr (S::NSTAGE == 2) static_for<g * NI / NSL, (g + 1) * NI / NSL>(item);
    };
    hs.mm_lds(st, lane, slice);
    if constexpr (WITH_OUT) {
      // O^T (this wave's d_v tiles x token tile nt) = S_c Q'^T + O_loc^T
#pragma unroll
      for (int ct = 0; ct < CT; ++ct)
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) pend[ct][nt] = raw4_to_f32(ops[u].ol[ct][nt]);
      // k-block outermost (4 x CT independent accumulators), reads one ahead
      constexpr int KB = DK / 32;
      const char *qs = st + S::NM_BYTES;
      Frag<T> q[2][4];
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) q[0][nt] = lds_frag<T>(qs, nt * KB, lane);
      static_for<0, KB>([&](auto kbc) {
        constexpr int kb = decltype(kbc)::value;
        if constexpr (kb + 1 < KB) {
#pragma unroll
          for (int nt = 0; nt < 4; ++nt) q[(kb + 1) & 1][nt] = lds_frag<T>(qs, nt * KB + kb + 1, lane);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
#pragma unroll
          for (int ct = 0; ct < CT; ++ct) pend[ct][nt] = mma(pend[ct][nt], hs.hb[ct][kb], q[kb & 1][nt]);
        slice(std::integral_constant<int, KB + kb>{});
        __builtin_amdgcn_sched_barrier(0);
      });
    }
    if constexpr (S::NSTAGE == 1) {
      __syncthreads();  // the single stage is free again
      static_for<0, NI>(item);
    }
  };
  // unrolled by two so the ring slots are compile-time; the odd last step
  // stays inside the loop (a separate tail copy would give the state a second
  // register assignment and a copy per iteration)
  for (int c = 0; c < nch; c += 2) {
    step(std::integral_constant<int, 0>{}, c);
    if (c + 1 < nch) step(std::integral_constant<int, 1>{}, c + 1);
  }
  if constexpr (WITH_OUT) out(nch - 1, pend);
}

// ------------------------------------------------------------- seg_transfer
template <typename T, int DK, int DV, bool KDA, bool APART>
__device__ __forceinline__ void transfer_part(const PrefillArgs &a, int s, int h, int4 sg, char *lds) {
  constexpr int NCOL = APART ? DK : DV;
  constexpr int CT = NCOL / 64, RT = DK / 16;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  HeadState<T, DK, NCOL> hs;
  // the first segment's B walk starts from the initial state (copied to s0c
  // for the first segment's state walk)
  const bool from_s0 = !APART && sg.w == 0 && a.s0;
  const size_t sbase = ((size_t)sg.x * a.Hv + h) * DK * DV;
#pragma unroll
  for (int ct = 0; ct < CT; ++ct)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int row = 16 * rt + 4 * grp + e;
        if (from_s0) {  // uniform for the workgroup
          const size_t i = sbase + (size_t)row * DV + dv_of(w * CT + ct, col);
          hs.H[ct][rt][e] = a.s0[i];
          a.s0c[i] = hs.H[ct][rt][e];
        } else {
          hs.H[ct][rt][e] = (APART && row == (w * CT + ct) * 16 + col) ? 1.f : 0.f;
        }
      }
  const int nch = sg.z;
  auto blk = [&](int c) { return (size_t)(sg.y + min(c, nch - 1)) * a.Hv + h; };
  auto no_out = [](int, const f32x4 (&)[CT][4]) {};
  walk_chunks<T, DK, NCOL, KDA, !APART, false>(hs, a, nch, blk, no_out, lds);

  const size_t mblk = (size_t)s * a.Hv + h;
  if constexpr (APART) {
    // A -> NM fragment order: lane (col', grp') of block (row tile rt, k-block
    // kb) holds A[16rt + col'][32kb + kmap(grp', j)], j = 0..7, i.e. columns
    // 32kb + 4grp' + 0..3 and 32kb + 16 + 4grp' + 0..3.  The accumulators hold
    // one column per lane, so A goes through LDS (row-major, padded rows).
    constexpr int LD = DK + 8;
    T *sA = reinterpret_cast<T *>(lds);
    __syncthreads();  // the walk's last stage reads are done
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int e = 0; e < 4; ++e)
          sA[(16 * rt + 4 * grp + e) * LD + (w * CT + ct) * 16 + col] = Elt<T>::from_f32(hs.H[ct][rt][e]);
    __syncthreads();
    T *am = static_cast<T *>(a.Aseg) + mblk * ((size_t)DK * DK);
    constexpr int NB = (DK / 16) * (DK / 32);  // operand blocks
    for (int b = w; b < NB; b += 4) {
      const int rt = b / (DK / 32), kb = b % (DK / 32);
      const T *row = sA + (16 * rt + col) * LD + 32 * kb + 4 * grp;
      float x[8];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        x[j] = Elt<T>::to_f32(row[j]);
        x[4 + j] = Elt<T>::to_f32(row[16 + j]);
      }
      store_frag_at(am + ((size_t)b * 64 + lane) * 8, make_frag<T>(x));
    }
  } else {
    float *bm = a.Bseg + mblk * ((size_t)DK * DV);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        store4(bm + ((size_t)((w * CT + ct) * RT + rt) * 64 + lane) * 4, hs.H[ct][rt]);
  }
}

template <typename T, int DK, int DV, bool KDA, bool SINGLE>
__global__ __launch_bounds__(kHeadThreads) void seg_transfer_kernel(PrefillArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  const int item = xcd_item(blockIdx.x, 2);  // (segment, head) x 2 parts
  const int pair = item >> 1, part = item & 1;
  if (pair >= a.max_segs * a.Hv) return;  // uniform for the workgroup
  const int s = pair / a.Hv, h = pair % a.Hv;
  const int4 sg = seg_info_at<SINGLE>(a, s);  // {sequence, first chunk, chunks, index in sequence}
  if (sg.x < 0) return;
  if (sg.w == seq_seg_at<SINGLE>(a, sg.x).y - 1) return;  // the last segment's map is never applied
  if (part == 0) {
    // the first segment needs no A: its B walk starts from the initial state
    if (sg.w == 0) return;
    transfer_part<T, DK, DV, KDA, true>(a, s, h, sg, lds);
  } else {
    transfer_part<T, DK, DV, KDA, false>(a, s, h, sg, lds);
  }
}

// ---------------------------------------------------------------- seg_state
// Applies the maps of segments j0 .. j1-1 to hs in order: H <- A H + B_seg.
template <typename T, int DK, int DV>
__device__ __forceinline__ void apply_maps(HeadState<T, DK, DV> &hs, const PrefillArgs &a, int j0, int j1, int h,
                                           char *lds) {
  using S = Stage<T, DK, false>;
  constexpr int CT = DV / 64, RT = DK / 16;
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  auto mblk = [&](int j) { return (size_t)min(j, j1 - 1) * a.Hv + h; };
  const char *Ag = static_cast<const char *>(a.Aseg);
  u32x4 sreg[S::NV];
  f32x4 bs[CT][RT];
  auto fetch_b = [&](int j) {
    const float *bm = a.Bseg + mblk(j) * ((size_t)DK * DV);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) bs[ct][rt] = load4(bm + ((size_t)((w * CT + ct) * RT + rt) * 64 + lane) * 4);
  };
  stage_fetch<S::NM_V>(sreg, Ag + mblk(j0) * S::NM_BYTES, nullptr, tid);
  fetch_b(j0);
  for (int j = j0; j < j1; ++j) {
    __syncthreads();  // every wave is done reading the previous map
    stage_put(sreg, lds, tid);
    stage_fetch<S::NM_V>(sreg, Ag + mblk(j + 1) * S::NM_BYTES, nullptr, tid);
    __syncthreads();
    hs.make_hb();
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) hs.H[ct][rt] = bs[ct][rt];
    fetch_b(j + 1);
    hs.mm_lds(lds, lane);
  }
  __syncthreads();  // the stage memory is reused by the walk
}

template <typename T, int DK, int DV, bool KDA, bool SINGLE>
__global__ __launch_bounds__(kHeadThreads) void seg_state_kernel(PrefillArgs a) {
  extern __shared__ __attribute__((aligned(16))) char lds[];
  constexpr int CT = DV / 64, RT = DK / 16;
  single_status<SINGLE>(a);
  const int pair = xcd_item(blockIdx.x, 1);
  if (pair >= a.max_segs * a.Hv) return;  // uniform for the workgroup
  const int s = pair / a.Hv, h = pair % a.Hv;
  const int4 sg = seg_info_at<SINGLE>(a, s);  // {sequence, first chunk, chunks, index in sequence}
  if (sg.x < 0) return;
  const int n = sg.x;
  const int4 si = seq_info_at<SINGLE>(a, n);  // {first chunk, chunks, start token, length}
  const int2 ss = seq_seg_at<SINGLE>(a, n);   // {first segment, segments}
  const int tid = threadIdx.x;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int nch = sg.z;

  HeadState<T, DK, DV> hs;
  const size_t sbase = ((size_t)n * a.Hv + h) * DK * DV;
  // state element of H[ct][rt][e]: row 16rt + 4grp + e, column dv_of(w CT + ct, col)
  auto sidx = [&](int ct, int rt, int e) {
    return sbase + (size_t)(16 * rt + 4 * grp + e) * DV + dv_of(w * CT + ct, col);
  };
  if (sg.w > 0) {
    // the first segment's B_seg is the state entering the second segment (its
    // walk started from s0); the maps of segments 1 .. sg.w - 1 follow
    const float *bm = a.Bseg + ((size_t)ss.x * a.Hv + h) * ((size_t)DK * DV);
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) hs.H[ct][rt] = load4(bm + ((size_t)((w * CT + ct) * RT + rt) * 64 + lane) * 4);
    if (ss.x + 1 < s) apply_maps(hs, a, ss.x + 1, s, h, lds);
  } else {
    // s0 itself only when this workgroup is the sequence's only writer of
    // s_final; otherwise the copy the segment maps made (s_final may alias s0)
    const float *src = a.s0 ? (ss.y > 1 ? a.s0c : a.s0) : nullptr;
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int e = 0; e < 4; ++e) hs.H[ct][rt][e] = src ? src[sidx(ct, rt, e)] : 0.f;
  }

  if (nch > 0) {
    const int tok0 = sg.w * a.seg_chunks * kChunk;  // first token of the segment inside its sequence
    // o rows of this segment: [si.z + tok0, si.z + min(len, tok0 + 64 nch)); rows
    // past the end (and the call for chunk -1) fall outside the buffer range
    const int rows = min(si.w - tok0, nch * kChunk);
    const size_t row_bytes = (size_t)a.Hv * DV * sizeof(T);
    const __amdgpu_buffer_rsrc_t orsrc =
        buffer_over(static_cast<T *>(a.o) + (size_t)(si.z + tok0) * a.Hv * DV, (uint32_t)(rows * row_bytes));
    auto blk = [&](int c) { return (size_t)(sg.y + min(c, nch - 1)) * a.Hv + h; };
    // pend[ct][nt][e]: o[token 16nt + col][dv_of(w CT + ct, 4grp + e)]; for a
    // tile pair (CT = 2) the two tiles' values are 8 consecutive columns
    auto out = [&](int c, const f32x4 (&pend)[CT][4]) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int r = c * kChunk + 16 * nt + col;  // row inside the segment (c may be -1)
        const int off = (int)((r * a.Hv + h) * DV) * (int)sizeof(T);
        if constexpr (CT == 2) {  // columns dv_of(2w, 4grp) .. +7
          store8_checked(orsrc, off + dv_of(2 * w, 4 * grp) * (int)sizeof(T), T{}, pend[0][nt] * a.scale,
                         pend[1][nt] * a.scale);
        } else {
#pragma unroll
          for (int ct = 0; ct < CT; ++ct)
            store4_checked(orsrc, off + dv_of(w * CT + ct, 4 * grp) * (int)sizeof(T), T{}, pend[ct][nt] * a.scale);
        }
      }
    };
    walk_chunks<T, DK, DV, KDA, true, true>(hs, a, nch, blk, out, lds);
  }

  if (a.s_final && sg.w == ss.y - 1) {
#pragma unroll
    for (int ct = 0; ct < CT; ++ct)
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int e = 0; e < 4; ++e) a.s_final[sidx(ct, rt, e)] = hs.H[ct][rt][e];
  }
}

// ------------------------------------------------------------------ launches
template <typename T, int DK, int DV>
static size_t transfer_lds() {
  using S = Stage<T, DK, false>;
  const size_t walk = (size_t)S::NSTAGE * S::BYTES;
  const size_t tr = (size_t)DK * (DK + 8) * sizeof(T);  // A transpose
  return walk > tr ? walk : tr;
}
template <typename T, int DK, int DV>
static size_t state_lds() {
  using S = Stage<T, DK, true>;
  return (size_t)S::NSTAGE * S::BYTES;  // >= one map stage
}

static long xcd_blocks(const PrefillArgs &a, int per_item) {
  const long items = (long)a.max_segs * a.Hv;
  const long groups = (items + kXcds - 1) / kXcds;
  return groups * kXcds * per_item;
}

template <typename T, int DK, int DV, bool KDA>
static hipError_t launch_transfer_t(const PrefillArgs &a, hipStream_t stream) {
  const size_t lds = transfer_lds<T, DK, DV>();
  auto kern = a.single ? seg_transfer_kernel<T, DK, DV, KDA, true> : seg_transfer_kernel<T, DK, DV, KDA, false>;
  hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)xcd_blocks(a, 2)), dim3(kHeadThreads), lds, stream, a);
  return hipGetLastError();
}

template <typename T, int DK, int DV, bool KDA>
static hipError_t launch_state_t(const PrefillArgs &a, hipStream_t stream) {
  const size_t lds = state_lds<T, DK, DV>();
  auto kern = a.single ? seg_state_kernel<T, DK, DV, KDA, true> : seg_state_kernel<T, DK, DV, KDA, false>;
  hipError_t e = hipFuncSetAttribute((const void *)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3((unsigned)xcd_blocks(a, 1)), dim3(kHeadThreads), lds, stream, a);
  return hipGetLastError();
}

template <typename T, bool KDA, bool TRANSFER>
static hipError_t dispatch_dims(const PrefillArgs &a, hipStream_t s) {
#define HAGDN_LAUNCH(dk, dv) \
  return TRANSFER ? launch_transfer_t<T, dk, dv, KDA>(a, s) : launch_state_t<T, dk, dv, KDA>(a, s)
  if (a.Dk == 64 && a.Dv == 64) HAGDN_LAUNCH(64, 64);
  if (a.Dk == 64 && a.Dv == 128) HAGDN_LAUNCH(64, 128);
  if (a.Dk == 128 && a.Dv == 64) HAGDN_LAUNCH(128, 64);
  HAGDN_LAUNCH(128, 128);
#undef HAGDN_LAUNCH
}

template <bool TRANSFER>
static hipError_t dispatch(const PrefillArgs &a, bool bf16, bool kda, hipStream_t s) {
  if (bf16) return kda ? dispatch_dims<bf16_t, true, TRANSFER>(a, s) : dispatch_dims<bf16_t, false, TRANSFER>(a, s);
  return kda ? dispatch_dims<float, true, TRANSFER>(a, s) : dispatch_dims<float, false, TRANSFER>(a, s);
}

hipError_t launch_seg_transfer(const PrefillArgs &a, bool bf16, bool kda, hipStream_t s) {
  if (bf16) return launch_seg_maps(a, kda, s);
  return kda ? dispatch_dims<float, true, true>(a, s) : dispatch_dims<float, false, true>(a, s);
}

hipError_t launch_seg_state(const PrefillArgs &a, bool bf16, bool kda, hipStream_t s) {
  return dispatch<false>(a, bf16, kda, s);
}

}  // namespace hagdn
