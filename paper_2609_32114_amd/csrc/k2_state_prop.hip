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

// Range-checked stores through a buffer resource over [base, base + bytes):
// lanes whose byte offset falls outside (negative ones included) store
// nothing, so the output store needs no branch -- a branch in the loop makes
// the compiler drain every in-flight load at the join.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t walk_buffer(void *base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)bytes, 0x00020000);  // gfx9 raw buffer word 3
}
__device__ __forceinline__ void walk_store4(__amdgpu_buffer_rsrc_t r, int off, bf16_t, f32x4 v) {
  typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
  u32x2 u;
  u[0] = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  u[1] = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  __builtin_amdgcn_raw_buffer_store_b64(u, r, off, 0, 0);
}
__device__ __forceinline__ void walk_store4(__amdgpu_buffer_rsrc_t r, int off, float, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, off, 0, 0);
}

// One chunk's state-independent operands for the rows one wave owns (the
// state update, on the critical path) ...
template <typename T, int DK, bool KDA>
struct StepOps {
  Frag<T> nm[2][DK / 32];         // NM rows 32w + 16i + col, k-block kb
  typename Raw4<T>::type b[2];    // B[32w + 16i + 4grp .. +3][dv]
  f32x4 dec[2];                   // decay of those rows (GDN: dec[0][0] only)
};
// ... and for the token tiles one wave outputs (off the critical path).
template <typename T, int DK>
struct OutOps {
  static constexpr int TPW = 4 / (DK / 32);  // output token tiles per wave
  Frag<T> qp[TPW][DK / 32];       // Q' block (token tile, kb): columns = tokens
  typename Raw4<T>::type ol[TPW]; // O_loc block (token tile, this d_v tile)
};

// Chunks of operands in flight: 3 for bf16 GDN, 2 for bf16 KDA (wider decay
// operands) and for fp32.  The bf16 depths fit the operand ring in 256
// architectural registers with no accumulation registers.  A deeper ring (4
// chunks) measured slower: it spills into accumulation registers, and the
// copies back land on the chain (workload of 1 x 4096 tokens, 16 heads: 53.2
// against 51.3 us).
template <typename T, bool KDA> constexpr int pipe_depth() {
  return sizeof(T) == 2 ? (KDA ? 2 : 3) : 2;
}

template <typename T, int DK, int DV, bool KDA, bool SINGLE>
__global__ __launch_bounds__(64 * (DK / 32), sizeof(T) == 2 ? 2 : 1) void state_prop_kernel(PrefillArgs a) {
  constexpr int NW = DK / 32;   // waves per chain
  constexpr int NT = DV / 16;   // d_v tiles per head
  constexpr int D = pipe_depth<T, KDA>();
  single_status<SINGLE>(a);
  const int b = blockIdx.x;
  const int xcd = b % kXcds, slot = b / kXcds;
  const int pair = (slot / NT) * kXcds + xcd;
  const int tile = slot % NT;
  if (pair >= a.N * a.Hv) return;  // uniform for the workgroup
  const int n = pair / a.Hv, h = pair % a.Hv;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int dv = dv_of(tile, col);  // state column this lane holds
  const int row0 = 32 * w;         // first state row of this wave
  const int4 si = seq_info_at<SINGLE>(a, n);  // {first chunk, chunks, start, length}
  const int nch = si.y;
  __shared__ Frag<T> xch[2][NW][64];  // S_c fragments, double-buffered by step parity

  // H[i][e] = S^T[row0 + 16i + 4grp + e][dv]
  f32x4 H[2];
  const size_t sbase = ((size_t)n * a.Hv + h) * DK * DV;
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      H[i][e] = a.s0 ? a.s0[sbase + (size_t)(row0 + 16 * i + 4 * grp + e) * DV + dv] : 0.f;

  if (nch > 0) {
    const T *__restrict__ NMg = static_cast<const T *>(a.NM);
    const T *__restrict__ Bg = static_cast<const T *>(a.Bc);
    const float *__restrict__ decg = a.dec;
    const T *__restrict__ Qpg = static_cast<const T *>(a.Qp);
    const T *__restrict__ Olg = static_cast<const T *>(a.Ol);
    // o rows of this sequence; rows past its end fall outside the buffer range
    const __amdgpu_buffer_rsrc_t orsrc = walk_buffer(static_cast<T *>(a.o) + (size_t)si.z * a.Hv * DV,
                                                     (uint32_t)((size_t)si.w * a.Hv * DV * sizeof(T)));
    // Operands of chunk c: block blk(c) (clamped into the sequence).  NM block
    // (row tile 2w+i, kb) in fragment order, B and O_loc lane-major (prefill.h).
    auto blk = [&](int c) { return (size_t)(si.x + min(c, nch - 1)) * a.Hv + h; };
    auto nm_at = [&](size_t b, int i, int kb) {
      return NMg + b * ((size_t)DK * DK) + ((size_t)((2 * w + i) * (DK / 32) + kb) * 64 + lane) * 8;
    };
    auto b_at = [&](size_t b, int i) {
      return Bg + b * ((size_t)DV * DK) + ((size_t)(tile * 64 + lane) * (DK / 16) + 2 * w + i) * 4;
    };
    auto qp_at = [&](size_t b, int u, int kb) {  // token tile nt = w + NW*u
      return Qpg + b * ((size_t)kChunk * DK) + ((size_t)((w + NW * u) * (DK / 32) + kb) * 64 + lane) * 8;
    };
    auto ol_at = [&](size_t b, int u) {
      return Olg + b * ((size_t)kChunk * DV) + ((size_t)(tile * 64 + lane) * 4 + w + NW * u) * 4;
    };
    auto load_dec = [&](StepOps<T, DK, KDA> &op, size_t b) {
      if constexpr (KDA) {
#pragma unroll
        for (int i = 0; i < 2; ++i) op.dec[i] = load4(decg + b * DK + row0 + 16 * i + 4 * grp);
      } else {
        op.dec[0][0] = decg[b * DK];
      }
    };
    auto load = [&](StepOps<T, DK, KDA> &op, int c) {
      const size_t b = blk(c);
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb) op.nm[i][kb] = load_frag_at(nm_at(b, i, kb));
        op.b[i] = load_raw4(b_at(b, i));
      }
      load_dec(op, b);
    };
    auto load_out = [&](OutOps<T, DK> &oq, int c) {
      const size_t b = blk(c);
#pragma unroll
      for (int u = 0; u < OutOps<T, DK>::TPW; ++u) {
#pragma unroll
        for (int kb = 0; kb < DK / 32; ++kb) oq.qp[u][kb] = load_frag_at(qp_at(b, u, kb));
        oq.ol[u] = load_raw4(ol_at(b, u));
      }
    };
    // output tiles of the previous chunk, stored one step late so the store
    // never waits on MFMA results inside the chain's critical path
    constexpr int TPW = OutOps<T, DK>::TPW;
    f32x4 pend[TPW];
    auto store_out = [&](int c) {
      const int base = c * kChunk;  // first token of chunk c inside the sequence
#pragma unroll
      for (int u = 0; u < TPW; ++u) {
        const int r = base + 16 * (w + NW * u) + col;
        walk_store4(orsrc, (int)(((size_t)r * a.Hv + h) * DV + dv_of(tile, 4 * grp)) * (int)sizeof(T), T{},
                    pend[u] * a.scale);
      }
    };
    // One chunk step.  Every operand register is refilled for chunk c + D right
    // after the instruction that consumes it, so the step's loads leave one or
    // two at a time behind matrix work instead of in a block that stalls the
    // wave at the address unit (each CU streams ~54 KiB per step from L2).
    auto step = [&](StepOps<T, DK, KDA> &op, OutOps<T, DK> &oq, int c) {
      const size_t bn = blk(c + D);
      // 5-read: this wave's k-block of S_c, published for the other waves
      const Frag<T> own = frag_from_acc<T>(H[0], H[1]);
      xch[c & 1][w][lane] = own;
      __syncthreads();
      Frag<T> hb[NW];
#pragma unroll
      for (int kb = 0; kb < NW; ++kb) hb[kb] = xch[c & 1][kb][lane];
      store_out(c - 1);  // chunk -1: every row falls outside the buffer range
      // 5-update: rows of S^T_{c+1} = D S^T_c + B + NM S^T_c (two accumulation
      // chains per tile, k-blocks split even/odd, summed at the end)
      f32x4 acc0[2], acc1[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const f32x4 d = KDA ? op.dec[i] : f32x4{op.dec[0][0], op.dec[0][0], op.dec[0][0], op.dec[0][0]};
        acc0[i] = d * H[i] + raw4_to_f32(op.b[i]);
        acc1[i] = zero4();
      }
#pragma unroll
      for (int i = 0; i < 2; ++i) op.b[i] = load_raw4(b_at(bn, i));
      load_dec(op, bn);
#pragma unroll
      for (int kb = 0; kb < NW; ++kb)
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          if (kb & 1) acc1[i] = mma(acc1[i], op.nm[i][kb], hb[kb]);
          else acc0[i] = mma(acc0[i], op.nm[i][kb], hb[kb]);
          op.nm[i][kb] = load_frag_at(nm_at(bn, i, kb));
        }
#pragma unroll
      for (int i = 0; i < 2; ++i) H[i] = acc0[i] + acc1[i];
      // operator #6 for token tile(s) w + NW*u: O^T = S_c Q'^T + O_loc^T (lane:
      // token col, d_v rows 4grp .. +3 of this tile); issued after the state
      // update so it runs while the next step converts and exchanges, stored
      // next step
#pragma unroll
      for (int u = 0; u < TPW; ++u) {
        pend[u] = raw4_to_f32(oq.ol[u]);
        oq.ol[u] = load_raw4(ol_at(bn, u));
#pragma unroll
        for (int kb = 0; kb < NW; ++kb) {
          pend[u] = mma(pend[u], hb[kb], oq.qp[u][kb]);
          oq.qp[u][kb] = load_frag_at(qp_at(bn, u, kb));
        }
      }
    };

    StepOps<T, DK, KDA> R[D];
    OutOps<T, DK> Q[D];
#pragma unroll
    for (int u = 0; u < D; ++u) {
      load(R[u], u);
      load_out(Q[u], u);
    }
    int c0 = 0;
    for (; c0 + D <= nch; c0 += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) step(R[u], Q[u], c0 + u);
    }
#pragma unroll
    for (int u = 0; u < D; ++u)
      if (c0 + u < nch) step(R[u], Q[u], c0 + u);  // uniform for the workgroup
    store_out(nch - 1);
  }

  if (a.s_final) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        a.s_final[sbase + (size_t)(row0 + 16 * i + 4 * grp + e) * DV + dv] = H[i][e];
  }
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
