// k2_walk.hip -- staged walks (bf16): the Reduce phase of chunkwise
// delta-rule prefill (paper Sec. 2.1, operator #5 H) with one wave per
// 16-column tile and the chunk's shared operands staged in LDS by a loader
// wave.  Two kernels:
//   state_walk_kernel  operators #5 and #6 over whole chains, for batches with
//                      more walks than CUs (k2_state_prop.hip walks the
//                      others, and every fp32 chain);
//   seg_pair_kernel,   the segment maps of the segment-parallel path (paper
//   seg_map_kernel     Sec. 4, Chunk-Seg-Seg; the rest of it is in
//                      k3_segments.hip): both maps of a segment in one
//                      workgroup when d_k = d_v, else one workgroup per map.
//
// Per chunk c the chunk-local kernel has left
//     S^T_{c+1} = D S^T_c + NM S^T_c + B,     O = scale (Q' S^T_c + O_loc)
// (prefill.h gives the block layouts).  Column split (paper Sec. 4,
// "Computation Splitting"): the d_v columns of S^T evolve independently, so a
// head splits into d_v/16 chains with no reduction between them.
//
// Workgroup -> work mapping is XCD-aware: consecutive workgroup ids are dealt
// round-robin to the 8 XCDs, so all workgroups of one (sequence, head) pair
// or (segment, head) pair share one XCD and its L2.
#include <atomic>
#include <type_traits>

#include "device.h"
#include "prefill.h"

namespace hagdn {
namespace {

constexpr int kXcds = 8;

__device__ __forceinline__ f32x4 raw4_to_f32(uint2 u) {
  f32x4 r;
  r[0] = __uint_as_float(u.x << 16);
  r[1] = __uint_as_float(u.x & 0xffff0000u);
  r[2] = __uint_as_float(u.y << 16);
  r[3] = __uint_as_float(u.y & 0xffff0000u);
  return r;
}
// Range-checked stores through a buffer resource over [base, base + bytes):
// lanes whose byte offset falls outside (negative ones included) store nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t walk_buffer(void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)bytes, 0x00020000);  // gfx9 raw buffer word 3
}
__device__ __forceinline__ void walk_store4(__amdgpu_buffer_rsrc_t r, int off, f32x4 v) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  u32x2 u;
  u[0] = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  u[1] = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  __builtin_amdgcn_raw_buffer_store_b64(u, r, off, 0, 0);
}

// ---------------------------------------------------------------------------
// Staged walk (bf16): one wave per 16-column tile holds all d_k rows of its
// tile, so a chain step is that wave's own products: no exchange between
// waves and no barrier between one step's state and the next step's
// products.  The chunk's NM and Q' blocks, read by every tile of the head,
// reach LDS through direct memory-to-LDS loads that a loader wave issues two
// chunks ahead into a three-stage ring; TPW tiles of one head share a
// workgroup and its stages.  Each tile wave fetches its own B and O_loc (and
// the GDN decay) into registers two chunks ahead.
//
// One step c of a tile wave: S_c as bf16 B fragments -> S <- D S + B -> o of
// chunk c-1 stored -> for each k-block kb: S += NM(:, kb) S_c(kb) and
// O^T += S_c(kb) Q'(:, kb)^T, with the NM fragments of k-block kb+1 read from
// LDS ahead of the products.  Before the last k-block comes the step's one
// barrier, B_(c+1): chunk c+1 has landed and every read of stage c is done
// (the loader then refills it), and chunk c+1's first fragments are read
// behind it while the last products run.
template <typename T, int DK, bool KDA, bool QP = true>
struct WalkStage {
  static constexpr int NM_BYTES = DK * DK * (int)sizeof(T);
  static constexpr int QP_BYTES = QP ? kChunk * DK * (int)sizeof(T) : 0;
  static constexpr int DEC_BYTES = KDA ? DK * 4 : 0;
  static constexpr int NM_OPS = NM_BYTES / 1024, QP_OPS = QP_BYTES / 1024;  // 16-byte lane loads
  static constexpr int DEC_OPS = DEC_BYTES / 256;                            // 4-byte lane loads
  static constexpr int OPS = NM_OPS + QP_OPS + DEC_OPS;  // loads per chunk
  static constexpr int BYTES = NM_BYTES + QP_BYTES + DEC_BYTES;
  static constexpr int NSTAGE = 3;
  static_assert(OPS < 64, "one chunk's loads fit the vector memory counter");
};

__device__ __forceinline__ void lds_load16(const void *g, unsigned char *l) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)l, 16, 0, 0);
}
__device__ __forceinline__ void lds_load4(const void *g, unsigned char *l) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void *)l, 4, 0, 0);
}
// s_waitcnt vmcnt(N) alone (export and LDS counters at their maxima; gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | 0x70 | 0xF00);
}
// Workgroup barrier that waits only for this wave's LDS operations; the fences
// keep the compiler from moving memory accesses across it.
__device__ __forceinline__ void walk_barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
}

template <typename T, int DK>
struct WalkLaneOps {
  uint2 b[DK / 16];  // B rows 16rt + 4grp .. +3 of this tile (raw bf16)
  uint2 ol[4];       // O_loc, token tile nt, d_v rows 4grp .. +3 of this tile
  float dec;         // GDN decay of the chunk
};

template <typename T, int DK, int DV, bool KDA, bool SINGLE, int TPW>
__global__ __launch_bounds__(64 * (TPW + 1), 1) void state_walk_kernel(PrefillArgs a) {
  static_assert(sizeof(T) == 2, "the staged walk is the bf16 path");
  using S = WalkStage<T, DK, KDA>;
  constexpr int RT = DK / 16, KB = DK / 32, NG = DV / (16 * TPW);
  extern __shared__ __align__(16) unsigned char lds[];
  single_status<SINGLE>(a);
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / NG) * kXcds + xcd;
  const int tg = slot % NG;
  if (pair >= a.N * a.Hv) return;  // uniform for the workgroup
  const int n = pair / a.Hv, h = pair % a.Hv;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int4 si = seq_info_at<SINGLE>(a, n);  // {first chunk, chunks, start, length}
  const int nch = si.y;
  auto blk = [&](int c) { return (size_t)(si.x + min(c, nch - 1)) * a.Hv + h; };

  if (wave == TPW) {
    // ---- loader wave: chunk c into stage c % 3, two chunks ahead
    if (nch > 0) {
      const unsigned char *NMg = static_cast<const unsigned char *>(a.NM);
      const unsigned char *QPg = static_cast<const unsigned char *>(a.Qp);
      auto issue = [&](int c) {
        const size_t bk = blk(c);
        unsigned char *st = lds + (c % S::NSTAGE) * S::BYTES;
        const unsigned char *nm = NMg + bk * S::NM_BYTES + lane * 16;
        const unsigned char *qp = QPg + bk * S::QP_BYTES + lane * 16;
#pragma unroll
        for (int j = 0; j < S::NM_OPS; ++j) lds_load16(nm + j * 1024, st + j * 1024);
#pragma unroll
        for (int j = 0; j < S::QP_OPS; ++j) lds_load16(qp + j * 1024, st + S::NM_BYTES + j * 1024);
        if constexpr (KDA) {
#pragma unroll
          for (int j = 0; j < S::DEC_OPS; ++j)
            lds_load4(a.dec + bk * DK + j * 64 + lane, st + S::NM_BYTES + S::QP_BYTES + j * 256);
        }
      };
      issue(0);
      issue(1);
      wait_vmcnt<S::OPS>();  // chunk 0 has landed
      walk_barrier();        // B_0
      for (int k = 1; k <= nch; ++k) {
        issue(k + 1);          // into the stage of chunk k - 2, whose reads ended before B_(k-1)
        wait_vmcnt<S::OPS>();  // chunk k has landed (chunk k + 1 may be in flight)
        walk_barrier();        // B_k
      }
      wait_vmcnt<0>();  // nothing in flight into LDS when the wave ends
    }
    return;
  }

  // ---- tile wave
  const int tile = tg * TPW + wave;
  const int col = lane & 15, grp = lane >> 4;
  const int dv = dv_of(tile, col);  // state column this lane holds
  f32x4 H[RT];                      // H[rt][e] = S^T[16rt + 4grp + e][dv]
  const size_t sbase = ((size_t)n * a.Hv + h) * DK * DV;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 4; ++e) H[rt][e] = a.s0 ? a.s0[sbase + (size_t)(16 * rt + 4 * grp + e) * DV + dv] : 0.f;

  if (nch > 0) {
    const T *__restrict__ Bg = static_cast<const T *>(a.Bc);
    const T *__restrict__ Olg = static_cast<const T *>(a.Ol);
    const __amdgpu_buffer_rsrc_t orsrc = walk_buffer(static_cast<T *>(a.o) + (size_t)si.z * a.Hv * DV,
                                                     (uint32_t)((size_t)si.w * a.Hv * DV * sizeof(T)));
    auto fetch = [&](WalkLaneOps<T, DK> &op, int c) {
      const size_t bk = blk(c);
      const T *bp = Bg + bk * ((size_t)DV * DK) + (size_t)(tile * 64 + lane) * (DK / 4);
#pragma unroll
      for (int i = 0; i < DK / 32; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(bp + 8 * i);
        op.b[2 * i] = make_uint2(v[0], v[1]);
        op.b[2 * i + 1] = make_uint2(v[2], v[3]);
      }
      const T *olp = Olg + bk * ((size_t)kChunk * DV) + (size_t)(tile * 64 + lane) * 16;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(olp + 8 * i);
        op.ol[2 * i] = make_uint2(v[0], v[1]);
        op.ol[2 * i + 1] = make_uint2(v[2], v[3]);
      }
      if constexpr (!KDA) op.dec = a.dec[bk * DK];
    };
    WalkLaneOps<T, DK> ring[2];
    fetch(ring[0], 0);
    fetch(ring[1], 1);
    f32x4 pend[4];  // O^T of a chunk: token tile nt, d_v rows 4grp .. +3
#pragma unroll
    for (int nt = 0; nt < 4; ++nt) pend[nt] = zero4();
    auto store_out = [&](int c) {
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) {
        const int r = c * kChunk + 16 * nt + col;  // chunk -1: outside the buffer range
        walk_store4(orsrc, (int)(((size_t)r * a.Hv + h) * DV + dv_of(tile, 4 * grp)) * (int)sizeof(T),
                    pend[nt] * a.scale);
      }
    };
    // NM fragments of one k-block (row tiles), read one k-block ahead; the
    // next chunk's first k-block is read behind the barrier that publishes
    // its stage, before this chunk's last products.  Q' fragments (token
    // tiles) are read at the start of their k-block and used after its NM
    // products.
    Frag<T> f[2][RT];
    auto read_nm = [&](const unsigned char *stl, int kb, int buf) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        f[buf][rt] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(stl + (rt * KB + kb) * 1024));
    };
    const unsigned char *lds_lane = lds + lane * 16;  // this lane's 16 bytes of every 1 KiB block
    walk_barrier();  // B_0: chunk 0 is in stage 0
    read_nm(lds_lane, 0, 0);
    auto step = [&](auto slot_c, int c) {
      constexpr int u = decltype(slot_c)::value;  // c & 1: operand ring slot
      // stage bases kept opaque so every read of a stage is one base register
      // plus an immediate offset
      const unsigned char *stl = lds_lane + __builtin_amdgcn_readfirstlane((c % S::NSTAGE) * S::BYTES);
      const unsigned char *stn = lds_lane + __builtin_amdgcn_readfirstlane(((c + 1) % S::NSTAGE) * S::BYTES);
      Frag<T> hb[KB];  // S_c, k-block kb: B operand of the update, A operand of the output
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) hb[kb] = frag_from_acc<T>(H[2 * kb], H[2 * kb + 1]);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        f32x4 d;
        if constexpr (KDA) {
          d = *reinterpret_cast<const f32x4 *>(stl - lane * 16 + S::NM_BYTES + S::QP_BYTES + (16 * rt + 4 * grp) * 4);
        } else {
          d = f32x4{ring[u].dec, ring[u].dec, ring[u].dec, ring[u].dec};
        }
        H[rt] = d * H[rt] + raw4_to_f32(ring[u].b[rt]);
      }
      store_out(c - 1);
#pragma unroll
      for (int nt = 0; nt < 4; ++nt) pend[nt] = raw4_to_f32(ring[u].ol[nt]);
      fetch(ring[u], c + 2);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int cur = kb & 1;
        Frag<T> q[4];
#pragma unroll
        for (int nt = 0; nt < 4; ++nt)
          q[nt] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(stl + S::NM_BYTES + (nt * KB + kb) * 1024));
        if (kb + 1 < KB) {
          read_nm(stl, kb + 1, cur ^ 1);
        } else {
          walk_barrier();            // B_(c+1): chunk c + 1 landed; every read of stage c done
          read_nm(stn, 0, cur ^ 1);  // KB is even: buffer 0
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) H[rt] = mma(H[rt], f[cur][rt], hb[kb]);
#pragma unroll
        for (int nt = 0; nt < 4; ++nt) pend[nt] = mma(pend[nt], hb[kb], q[nt]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    for (int c = 0; c < nch; c += 2) {
      step(std::integral_constant<int, 0>{}, c);
      if (c + 1 < nch) step(std::integral_constant<int, 1>{}, c + 1);  // uniform for the workgroup
    }
    store_out(nch - 1);
  }

  if (a.s_final) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int e = 0; e < 4; ++e) a.s_final[sbase + (size_t)(16 * rt + 4 * grp + e) * DV + dv] = H[rt][e];
  }
}


// ---------------------------------------------------------------------------
// Segment maps on the staged walk (bf16; the Chunk-Seg-Seg path, paper Sec. 4):
// the chunk maps of one segment composed, S^T_out = A S^T_in + B_seg.  A is the
// walk of the d_k x d_k identity through the segment's chunks without their B
// terms, B_seg the walk of a zero state with them; both are column tiles, so
// each tile wave walks one 16-column tile of A or of B_seg and a loader wave
// stages the chunks' NM blocks (shared by every tile) as above.  Workgroups of
// TPW tiles: d_k / (16 TPW) of them for A, then d_v / (16 TPW) for B_seg, all
// on one XCD.  Only segments that another segment of the same sequence
// follows get a map, and the first segment has no A: its B_seg walk starts
// from the initial state (copied to s0c on the way, prefill.h).  A is stored in NM's fragment order (bf16) through an LDS transpose,
// B_seg in fp32 in the state kernel's tile order (prefill.h).
template <typename T, int DK, int DV, bool KDA, bool SINGLE, int TPW>
__global__ __launch_bounds__(64 * (TPW + 1), 1) void seg_map_kernel(PrefillArgs a) {
  static_assert(sizeof(T) == 2, "the staged walk is the bf16 path");
  static_assert(TPW % 2 == 0, "A's fragment blocks pair adjacent column tiles");
  using S = WalkStage<T, DK, KDA, false>;
  constexpr int RT = DK / 16, KB = DK / 32;
  constexpr int NA = DK / (16 * TPW), NB = DV / (16 * TPW);  // workgroups per map
  extern __shared__ __align__(16) unsigned char lds[];
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / (NA + NB)) * kXcds + xcd;  // (segment, value head)
  const int part = slot % (NA + NB);                  // < NA: A, else B_seg
  if (pair >= a.max_segs * a.Hv) return;  // uniform for the workgroup
  const int sgi = pair / a.Hv, h = pair % a.Hv;
  const int4 sg = seg_info_at<SINGLE>(a, sgi);  // {sequence, first chunk, chunks, index in sequence}
  if (sg.x < 0) return;
  if (sg.w == seq_seg_at<SINGLE>(a, sg.x).y - 1) return;  // the last segment's map is never applied
  const bool apart = part < NA;
  if (apart && sg.w == 0) return;  // the first segment's B walk starts from s0 instead
  const int nch = sg.z;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  auto blk = [&](int c) { return (size_t)(sg.y + min(c, nch - 1)) * a.Hv + h; };

  if (wave == TPW) {
    // ---- loader wave: chunk c into stage c % 3, two chunks ahead
    if (nch > 0) {
      const unsigned char *NMg = static_cast<const unsigned char *>(a.NM);
      auto issue = [&](int c) {
        const size_t bk = blk(c);
        unsigned char *st = lds + (c % S::NSTAGE) * S::BYTES;
        const unsigned char *nm = NMg + bk * S::NM_BYTES + lane * 16;
#pragma unroll
        for (int j = 0; j < S::NM_OPS; ++j) lds_load16(nm + j * 1024, st + j * 1024);
        if constexpr (KDA) {
#pragma unroll
          for (int j = 0; j < S::DEC_OPS; ++j) lds_load4(a.dec + bk * DK + j * 64 + lane, st + S::NM_BYTES + j * 256);
        }
      };
      issue(0);
      issue(1);
      wait_vmcnt<S::OPS>();  // chunk 0 has landed
      walk_barrier();        // B_0
      for (int k = 1; k <= nch; ++k) {
        issue(k + 1);          // into the stage of chunk k - 2, whose reads ended before B_(k-1)
        wait_vmcnt<S::OPS>();  // chunk k has landed (chunk k + 1 may be in flight)
        walk_barrier();        // B_k
      }
      wait_vmcnt<0>();  // nothing in flight into LDS when the wave ends
    }
    walk_barrier();  // B_end: the tile waves' transpose may reuse the stages
    return;
  }

  // ---- tile wave: column tile t of A (plain column indices 16t ..) or of
  //      B_seg (the state's columns dv_of(t, ..))
  const int t = (apart ? part : part - NA) * TPW + wave;
  const int col = lane & 15, grp = lane >> 4;
  f32x4 H[RT];
  // the first segment's B walk starts from the initial state, copied to s0c
  const bool from_s0 = !apart && sg.w == 0 && a.s0;
  const size_t sbase = ((size_t)sg.x * a.Hv + h) * DK * DV;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 16 * rt + 4 * grp + e;
      if (from_s0) {  // uniform for the workgroup
        const size_t i = sbase + (size_t)row * DV + dv_of(t, col);
        H[rt][e] = a.s0[i];
        a.s0c[i] = H[rt][e];
      } else {
        H[rt][e] = (apart && row == 16 * t + col) ? 1.f : 0.f;
      }
    }

  if (nch > 0) {
    const T *__restrict__ Bg = static_cast<const T *>(a.Bc);
    struct Lane {
      uint2 b[RT];  // B rows 16rt + 4grp .. +3 of tile t (B_seg walks only)
      float dec;    // GDN decay of the chunk
    };
    auto fetch = [&](Lane &op, int c) {
      const size_t bk = blk(c);
      if (!apart) {
        const T *bp = Bg + bk * ((size_t)DV * DK) + (size_t)(t * 64 + lane) * (DK / 4);
#pragma unroll
        for (int i = 0; i < DK / 32; ++i) {
          const u32x4 v = *reinterpret_cast<const u32x4 *>(bp + 8 * i);
          op.b[2 * i] = make_uint2(v[0], v[1]);
          op.b[2 * i + 1] = make_uint2(v[2], v[3]);
        }
      } else {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) op.b[rt] = make_uint2(0u, 0u);
      }
      if constexpr (!KDA) op.dec = a.dec[bk * DK];
    };
    Lane ring[2];
    fetch(ring[0], 0);
    fetch(ring[1], 1);
    Frag<T> f[2][RT];
    auto read_nm = [&](const unsigned char *stl, int kb, int buf) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        f[buf][rt] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(stl + (rt * KB + kb) * 1024));
    };
    const unsigned char *lds_lane = lds + lane * 16;
    walk_barrier();  // B_0: chunk 0 is in stage 0
    read_nm(lds_lane, 0, 0);
    auto step = [&](auto slot_c, int c) {
      constexpr int u = decltype(slot_c)::value;  // c & 1: operand ring slot
      const unsigned char *stl = lds_lane + __builtin_amdgcn_readfirstlane((c % S::NSTAGE) * S::BYTES);
      const unsigned char *stn = lds_lane + __builtin_amdgcn_readfirstlane(((c + 1) % S::NSTAGE) * S::BYTES);
      Frag<T> hb[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) hb[kb] = frag_from_acc<T>(H[2 * kb], H[2 * kb + 1]);
      f32x4 dk[KDA ? RT : 1];
      if constexpr (KDA) {
#pragma unroll
        for (int rt = 0; rt < RT; ++rt)
          dk[rt] = *reinterpret_cast<const f32x4 *>(stl - lane * 16 + S::NM_BYTES + (16 * rt + 4 * grp) * 4);
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const f32x4 d = KDA ? dk[KDA ? rt : 0] : f32x4{ring[u].dec, ring[u].dec, ring[u].dec, ring[u].dec};
        H[rt] = d * H[rt] + raw4_to_f32(ring[u].b[rt]);
      }
      fetch(ring[u], c + 2);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int cur = kb & 1;
        if (kb + 1 < KB) {
          read_nm(stl, kb + 1, cur ^ 1);
        } else {
          walk_barrier();            // B_(c+1): chunk c + 1 landed; every read of stage c done
          read_nm(stn, 0, cur ^ 1);  // KB is even: buffer 0
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) H[rt] = mma(H[rt], f[cur][rt], hb[kb]);
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    for (int c = 0; c < nch; c += 2) {
      step(std::integral_constant<int, 0>{}, c);
      if (c + 1 < nch) step(std::integral_constant<int, 1>{}, c + 1);  // uniform for the workgroup
    }
  }
  walk_barrier();  // B_end: every stage read and every load landed

  const size_t mblk = (size_t)sgi * a.Hv + h;
  if (!apart) {
    float *bm = a.Bseg + mblk * ((size_t)DK * DV);
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
      *reinterpret_cast<f32x4 *>(bm + ((size_t)(t * RT + rt) * 64 + lane) * 4) = H[rt];
    return;
  }
  // A: this workgroup's 16 TPW columns, rounded to bf16, row-major in LDS
  // (rows padded by 8 elements), then stored as NM-ordered operand blocks
  // (row tile rt, k-block kb): slot j of lane (col, grp) holds
  // A[16rt + col][32kb + kmap(grp, j)]
  constexpr int LD = 16 * TPW + 8;
  T *sA = reinterpret_cast<T *>(lds);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 4; ++e) sA[(16 * rt + 4 * grp + e) * LD + 16 * wave + col] = Elt<T>::from_f32(H[rt][e]);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  T *am = static_cast<T *>(a.Aseg) + mblk * ((size_t)DK * DK);
  constexpr int KBW = TPW / 2;        // k-blocks of this workgroup
  const int kb0 = part * KBW;         // first k-block of this workgroup
  for (int q = wave; q < RT * KBW; q += TPW) {
    const int rt = q / KBW, kbl = q % KBW;
    const T *row = sA + (16 * rt + col) * LD + 32 * kbl + 4 * grp;
    float x[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = Elt<T>::to_f32(row[j]);
      x[4 + j] = Elt<T>::to_f32(row[16 + j]);
    }
    store_frag_at(am + ((size_t)(rt * KB + kb0 + kbl) * 64 + lane) * 8, make_frag<T>(x));
  }
}

// Both maps of a segment in one workgroup (d_k = d_v = D): wave w walks
// column tile w of A and column tile w of B_seg side by side, so every NM
// fragment it reads from LDS feeds two products and each NM block crosses
// the CU once per step.  With D/16 waves of about 200 registers a loader wave
// would not fit beside them, so the waves issue the stage loads themselves
// (load j by wave j mod D/16), as the last memory operations of a step, and
// wait for their share of the next chunk before its barrier.
template <typename T, int D, bool KDA, bool SINGLE>
__global__ __launch_bounds__(64 * (D / 16), 1) void seg_pair_kernel(PrefillArgs a) {
  static_assert(sizeof(T) == 2, "the staged walk is the bf16 path");
  using S = WalkStage<T, D, KDA, false>;
  constexpr int NW = D / 16, RT = D / 16, KB = D / 32;
  constexpr int SHARE = S::OPS / NW;  // fewest stage loads of one wave per chunk
  extern __shared__ __align__(16) unsigned char lds[];
  const int pair = blockIdx.x;  // (segment, value head): nothing shared between workgroups
  if (pair >= a.max_segs * a.Hv) return;  // uniform for the workgroup
  const int sgi = pair / a.Hv, h = pair % a.Hv;
  const int4 sg = seg_info_at<SINGLE>(a, sgi);  // {sequence, first chunk, chunks, index in sequence}
  if (sg.x < 0) return;
  if (sg.w == seq_seg_at<SINGLE>(a, sg.x).y - 1) return;  // the last segment's map is never applied
  const bool do_a = sg.w > 0;  // the first segment's B walk starts from s0 instead
  const int nch = sg.z;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  auto blk = [&](int c) { return (size_t)(sg.y + min(c, nch - 1)) * a.Hv + h; };
  const unsigned char *NMg = static_cast<const unsigned char *>(a.NM);
  auto issue_share = [&](int c) {
    const size_t bk = blk(c);
    unsigned char *st = lds + (c % S::NSTAGE) * S::BYTES;
    for (int j = w; j < S::OPS; j += NW) {  // uniform for the wave
      if (j < S::NM_OPS) {
        lds_load16(NMg + bk * S::NM_BYTES + lane * 16 + j * 1024, st + j * 1024);
      } else {
        const int q = j - S::NM_OPS;
        lds_load4(a.dec + bk * D + q * 64 + lane, st + S::NM_BYTES + q * 256);
      }
    }
  };

  f32x4 HA[RT], HB[RT];  // tile w of A (columns 16w + col) and of B_seg (columns dv_of(w, col))
  // the first segment's B walk starts from the initial state, copied to s0c
  const bool from_s0 = sg.w == 0 && a.s0;
  const size_t sbase = ((size_t)sg.x * a.Hv + h) * D * D;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int row = 16 * rt + 4 * grp + e;
      HA[rt][e] = (row == 16 * w + col) ? 1.f : 0.f;
      if (from_s0) {  // uniform for the workgroup
        const size_t i = sbase + (size_t)row * D + dv_of(w, col);
        HB[rt][e] = a.s0[i];
        a.s0c[i] = HB[rt][e];
      } else {
        HB[rt][e] = 0.f;
      }
    }

  if (nch > 0) {
    const T *__restrict__ Bg = static_cast<const T *>(a.Bc);
    struct Lane {
      uint2 b[RT];  // B rows 16rt + 4grp .. +3 of tile w
      float dec;    // GDN decay of the chunk
    };
    auto fetch = [&](Lane &op, int c) {
      const size_t bk = blk(c);
      const T *bp = Bg + bk * ((size_t)D * D) + (size_t)(w * 64 + lane) * (D / 4);
#pragma unroll
      for (int i = 0; i < D / 32; ++i) {
        const u32x4 v = *reinterpret_cast<const u32x4 *>(bp + 8 * i);
        op.b[2 * i] = make_uint2(v[0], v[1]);
        op.b[2 * i + 1] = make_uint2(v[2], v[3]);
      }
      if constexpr (!KDA) op.dec = a.dec[bk * D];
    };
    Lane ring[2];
    fetch(ring[0], 0);
    fetch(ring[1], 1);
    __builtin_amdgcn_sched_barrier(0);
    issue_share(0);
    issue_share(1);
    __builtin_amdgcn_sched_barrier(0);
    wait_vmcnt<SHARE>();  // this wave's share of chunk 0 has landed
    Frag<T> f[2][RT];
    auto read_nm = [&](const unsigned char *stl, int kb, int buf) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
        f[buf][rt] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4 *>(stl + (rt * KB + kb) * 1024));
    };
    const unsigned char *lds_lane = lds + lane * 16;
    walk_barrier();  // B_0: chunk 0 is in stage 0
    read_nm(lds_lane, 0, 0);
    auto step = [&](auto slot_c, int c) {
      constexpr int u = decltype(slot_c)::value;  // c & 1: operand ring slot
      const unsigned char *stl = lds_lane + __builtin_amdgcn_readfirstlane((c % S::NSTAGE) * S::BYTES);
      const unsigned char *stn = lds_lane + __builtin_amdgcn_readfirstlane(((c + 1) % S::NSTAGE) * S::BYTES);
      Frag<T> ha[KB], hb[KB];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        ha[kb] = frag_from_acc<T>(HA[2 * kb], HA[2 * kb + 1]);
        hb[kb] = frag_from_acc<T>(HB[2 * kb], HB[2 * kb + 1]);
      }
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        f32x4 d;
        if constexpr (KDA) {
          d = *reinterpret_cast<const f32x4 *>(stl - lane * 16 + S::NM_BYTES + (16 * rt + 4 * grp) * 4);
        } else {
          d = f32x4{ring[u].dec, ring[u].dec, ring[u].dec, ring[u].dec};
        }
        HA[rt] = d * HA[rt];
        HB[rt] = d * HB[rt] + raw4_to_f32(ring[u].b[rt]);
      }
      fetch(ring[u], c + 2);
      // this wave's share of chunk c + 2, into the stage step c - 1 read: the
      // last memory operations of the step, so that the wait below leaves
      // only them in flight
      __builtin_amdgcn_sched_barrier(0);
      issue_share(c + 2);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int cur = kb & 1;
        if (kb + 1 < KB) {
          read_nm(stl, kb + 1, cur ^ 1);
        } else {
          wait_vmcnt<SHARE>();       // this wave's share of chunk c + 1 has landed
          walk_barrier();            // B_(c+1): chunk c + 1 landed; every read of stage c done
          read_nm(stn, 0, cur ^ 1);  // KB is even: buffer 0
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          HA[rt] = mma(HA[rt], f[cur][rt], ha[kb]);
          HB[rt] = mma(HB[rt], f[cur][rt], hb[kb]);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    };
    for (int c = 0; c < nch; c += 2) {
      step(std::integral_constant<int, 0>{}, c);
      if (c + 1 < nch) step(std::integral_constant<int, 1>{}, c + 1);  // uniform for the workgroup
    }
    wait_vmcnt<0>();  // nothing in flight into LDS
  }
  walk_barrier();  // B_end: every stage read and every load landed

  const size_t mblk = (size_t)sgi * a.Hv + h;
  float *bm = a.Bseg + mblk * ((size_t)D * D);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) *reinterpret_cast<f32x4 *>(bm + ((size_t)(w * RT + rt) * 64 + lane) * 4) = HB[rt];
  if (!do_a) return;  // uniform for the workgroup
  // A rounded to bf16, row-major in LDS (rows padded by 8 elements), then
  // stored as NM-ordered operand blocks (row tile rt, k-block kb): slot j of
  // lane (col, grp) holds A[16rt + col][32kb + kmap(grp, j)]
  constexpr int LD = D + 8;
  T *sA = reinterpret_cast<T *>(lds);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int e = 0; e < 4; ++e) sA[(16 * rt + 4 * grp + e) * LD + 16 * w + col] = Elt<T>::from_f32(HA[rt][e]);
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "workgroup");
  T *am = static_cast<T *>(a.Aseg) + mblk * ((size_t)D * D);
  for (int q = w; q < RT * KB; q += NW) {
    const int rt = q / KB, kb = q % KB;
    const T *row = sA + (16 * rt + col) * LD + 32 * kb + 4 * grp;
    float x[8];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      x[j] = Elt<T>::to_f32(row[j]);
      x[4 + j] = Elt<T>::to_f32(row[16 + j]);
    }
    store_frag_at(am + ((size_t)(rt * KB + kb) * 64 + lane) * 8, make_frag<T>(x));
  }
}

template <typename T, int D, bool KDA, bool SINGLE>
static hipError_t launch_pair_t(const PrefillArgs &a, hipStream_t stream) {
  using S = WalkStage<T, D, KDA, false>;
  constexpr int kMaxDevices = 64;
  static std::atomic<bool> done[kMaxDevices];
  const void *kern = reinterpret_cast<const void *>(&seg_pair_kernel<T, D, KDA, SINGLE>);
  constexpr int walk_lds = S::NSTAGE * S::BYTES;
  constexpr int tr_lds = D * (D + 8) * (int)sizeof(T);
  const int lds = walk_lds > tr_lds ? walk_lds : tr_lds;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices || !done[dev].load(std::memory_order_relaxed)) {
    if ((e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds)) != hipSuccess) return e;
    if (dev >= 0 && dev < kMaxDevices) done[dev].store(true, std::memory_order_relaxed);
  }
  const long blocks = (long)a.max_segs * a.Hv;
  hipLaunchKernelGGL((seg_pair_kernel<T, D, KDA, SINGLE>), dim3((unsigned)blocks), dim3(64 * (D / 16)), lds, stream,
                     a);
  return hipGetLastError();
}

template <typename T, int DK, int DV, bool KDA, bool SINGLE, int TPW>
static hipError_t launch_maps_t(const PrefillArgs &a, hipStream_t stream) {
  using S = WalkStage<T, DK, KDA, false>;
  constexpr int kMaxDevices = 64;
  static std::atomic<bool> done[kMaxDevices];
  const void *kern = reinterpret_cast<const void *>(&seg_map_kernel<T, DK, DV, KDA, SINGLE, TPW>);
  constexpr int walk_lds = S::NSTAGE * S::BYTES;
  constexpr int tr_lds = DK * (16 * TPW + 8) * (int)sizeof(T);
  const int lds = walk_lds > tr_lds ? walk_lds : tr_lds;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices || !done[dev].load(std::memory_order_relaxed)) {
    if ((e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds)) != hipSuccess) return e;
    if (dev >= 0 && dev < kMaxDevices) done[dev].store(true, std::memory_order_relaxed);
  }
  const long items = (long)a.max_segs * a.Hv;
  const long groups = (items + kXcds - 1) / kXcds;
  const long blocks = groups * kXcds * (DK / (16 * TPW) + DV / (16 * TPW));
  hipLaunchKernelGGL((seg_map_kernel<T, DK, DV, KDA, SINGLE, TPW>), dim3((unsigned)blocks), dim3(64 * (TPW + 1)), lds,
                     stream, a);
  return hipGetLastError();
}

template <int DK, int DV, bool KDA>
hipError_t launch_maps_dims(const PrefillArgs &a, hipStream_t s) {
  if constexpr (DK == DV)
    return a.single ? launch_pair_t<bf16_t, DK, KDA, true>(a, s) : launch_pair_t<bf16_t, DK, KDA, false>(a, s);
  // as many tiles per workgroup as the narrower map has: fewer copies of each NM block
  constexpr int TPW = (DK < DV ? DK : DV) / 16;
  return a.single ? launch_maps_t<bf16_t, DK, DV, KDA, true, TPW>(a, s)
                  : launch_maps_t<bf16_t, DK, DV, KDA, false, TPW>(a, s);
}

template <bool KDA>
hipError_t launch_maps_kind(const PrefillArgs &a, hipStream_t s) {
  if (a.Dk == 64 && a.Dv == 64) return launch_maps_dims<64, 64, KDA>(a, s);
  if (a.Dk == 64 && a.Dv == 128) return launch_maps_dims<64, 128, KDA>(a, s);
  if (a.Dk == 128 && a.Dv == 64) return launch_maps_dims<128, 64, KDA>(a, s);
  return launch_maps_dims<128, 128, KDA>(a, s);
}

// The staged walk's LDS (three stages) exceeds the default 64 KiB limit: raise
// it once per device and instance.
template <typename T, int DK, int DV, bool KDA, bool SINGLE, int TPW>
static hipError_t launch_walk_t(const PrefillArgs &a, long groups, hipStream_t stream) {
  using S = WalkStage<T, DK, KDA>;
  constexpr int kMaxDevices = 64;
  static std::atomic<bool> done[kMaxDevices];
  const void *kern = reinterpret_cast<const void *>(&state_walk_kernel<T, DK, DV, KDA, SINGLE, TPW>);
  const int lds = S::NSTAGE * S::BYTES;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices || !done[dev].load(std::memory_order_relaxed)) {
    if ((e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, lds)) != hipSuccess) return e;
    if (dev >= 0 && dev < kMaxDevices) done[dev].store(true, std::memory_order_relaxed);
  }
  const long blocks = groups * kXcds * (DV / (16 * TPW));
  hipLaunchKernelGGL((state_walk_kernel<T, DK, DV, KDA, SINGLE, TPW>), dim3((unsigned)blocks), dim3(64 * (TPW + 1)),
                     lds, stream, a);
  return hipGetLastError();
}

template <typename T, int DK, int DV, bool KDA, int TPW>
static hipError_t launch_walk_single(const PrefillArgs &a, long groups, hipStream_t stream) {
  return a.single ? launch_walk_t<T, DK, DV, KDA, true, TPW>(a, groups, stream)
                  : launch_walk_t<T, DK, DV, KDA, false, TPW>(a, groups, stream);
}

template <int DK, int DV, bool KDA>
hipError_t launch_walk_dims(const PrefillArgs &a, int cus, hipStream_t stream) {
  const long pairs = (long)a.N * a.Hv;
  const long groups = (pairs + kXcds - 1) / kXcds;
  const long blocks = groups * kXcds * (DV / 16);
  // tiles of a head share a workgroup and its stages: two while that fits
  // the CUs in one round, else four
  if (blocks <= 2L * cus) return launch_walk_single<bf16_t, DK, DV, KDA, 2>(a, groups, stream);
  return launch_walk_single<bf16_t, DK, DV, KDA, 4>(a, groups, stream);
}

template <bool KDA>
hipError_t launch_walk_kind(const PrefillArgs &a, int cus, hipStream_t s) {
  if (a.Dk == 64 && a.Dv == 64) return launch_walk_dims<64, 64, KDA>(a, cus, s);
  if (a.Dk == 64 && a.Dv == 128) return launch_walk_dims<64, 128, KDA>(a, cus, s);
  if (a.Dk == 128 && a.Dv == 64) return launch_walk_dims<128, 64, KDA>(a, cus, s);
  return launch_walk_dims<128, 128, KDA>(a, cus, s);
}

}  // namespace

hipError_t launch_seg_maps(const PrefillArgs &a, bool kda, hipStream_t s) {
  return kda ? launch_maps_kind<true>(a, s) : launch_maps_kind<false>(a, s);
}

hipError_t launch_state_walk(const PrefillArgs &a, bool kda, int cus, hipStream_t s) {
  return kda ? launch_walk_kind<true>(a, cus, s) : launch_walk_kind<false>(a, cus, s);
}

}  // namespace hagdn
