// state_walk.h -- the whole-chain state walk of one (sequence, value head,
// d_v tile): operator #5 (H) over every chunk of the sequence, fused with
// operator #6 (O).  Used by the state kernel (k2_state_prop.hip) and by the
// overlapped chunk-local launch (k1_chunk_local.hip).
#pragma once

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
  int ready;                      // overlapped walk: ready flag of the chunk this slot loads next
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

// Ready-flag polling of an overlapped walk.  A flag is read with an
// agent-scope atomic load (global_load sc1), which skips the CU's L1 and is
// served by this XCD's L2 -- where the chunk-local blocks of this head stored
// their factors and then set the flag with an atomic.  A workgroup-scope load
// (sc0) was served from the L1 and kept returning the first value it read; an
// atomic read-modify-write works too but cost the walk ~10 % per step.
// Between polls a wave sleeps kOvlSleep x 64 cycles; after kOvlMaxPolls polls
// it stops waiting and reports HAGDN_DEV_WAIT_TIMEOUT.
constexpr int kOvlSleep = 8;
constexpr int kOvlMaxPolls = 1 << 21;

// The walk's LDS: 2 x NW x 64 fragments.  A walk workgroup of the overlapped
// launch uses the start of the launch's dynamic LDS, which its chunk-local
// workgroups use for their own tiles (a workgroup has one role), so the
// launch asks for no LDS beyond the chunk-local kernel's.
template <typename T, int NW, bool DYN>
__device__ __forceinline__ Frag<T> (&walk_exchange())[2][NW][64] {
  if constexpr (DYN) {
    extern __shared__ __align__(16) unsigned char walk_dyn_lds[];
    return *reinterpret_cast<Frag<T>(*)[2][NW][64]>(walk_dyn_lds);
  } else {
    __shared__ Frag<T> xch[2][NW][64];
    return xch;
  }
}

// Walk of one (sequence, value head) pair's d_v tile `tile` by one workgroup
// of DK/32 waves (xch: DK/32 x 64 fragments of LDS, double-buffered).  OVL:
// the chunk-local kernel runs at the same time in the same launch, and the
// walk waits for each chunk's ready flag before it loads the chunk's factors
// (ovl_wait below).
template <typename T, int DK, int DV, bool KDA, bool SINGLE, bool OVL>
__device__ __forceinline__ void walk_tile(const PrefillArgs &a, int pair, int tile) {
  constexpr int NW = DK / 32;   // waves per chain
  constexpr int D = pipe_depth<T, KDA>();
  const int n = pair / a.Hv, h = pair % a.Hv;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int col = lane & 15, grp = lane >> 4;
  const int dv = dv_of(tile, col);  // state column this lane holds
  const int row0 = 32 * w;         // first state row of this wave
  const int4 si = seq_info_at<SINGLE>(a, n);  // {first chunk, chunks, start, length}
  const int nch = si.y;
  // S_c fragments, double-buffered by step parity
  Frag<T>(&xch)[2][NW][64] = walk_exchange<T, NW, OVL>();

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
    // Overlapped launch: a chunk's factors are loaded only once its ready flag
    // is set.  Each ring slot carries the flag of the chunk it loads next,
    // read D steps ahead (so waiting for it waits only for older loads, which
    // the pipeline has consumed by then); a flag still clear is polled until
    // it is set or the polls run out (timed_out: the walk goes on, reports
    // HAGDN_DEV_WAIT_TIMEOUT and waits no more).
    bool timed_out = false;
    int *const flags = a.ovl + kOvlFlags;
    auto ovl_flag = [&](int c) {
      return __hip_atomic_load(flags + blk(c), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    };
    auto ovl_wait = [&](int flag, int c) {
      int v = __builtin_amdgcn_readfirstlane(flag);
      if (v == 0 && !timed_out) {  // uniform for the wave
        for (int polls = 0; v == 0 && polls < kOvlMaxPolls; ++polls) {
          __builtin_amdgcn_s_sleep(kOvlSleep);
          v = __builtin_amdgcn_readfirstlane(ovl_flag(c));
        }
        timed_out = v == 0;
      }
    };
    // One chunk step.  Every operand register is refilled for chunk c + D right
    // after the instruction that consumes it, so the step's loads leave one or
    // two at a time behind matrix work instead of in a block that stalls the
    // wave at the address unit (each CU streams ~54 KiB per step from L2).
    auto step = [&](StepOps<T, DK, KDA> &op, OutOps<T, DK> &oq, int c) {
      const size_t bn = blk(c + D);
      if constexpr (OVL) {  // chunk c + D is loaded below: its flag, read D steps ago
        ovl_wait(op.ready, c + D);
        op.ready = ovl_flag(c + 2 * D);
      }
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
    if constexpr (OVL) {
#pragma unroll
      for (int u = 0; u < D; ++u) {
        R[u].ready = ovl_flag(u);
        ovl_wait(R[u].ready, u);
        R[u].ready = ovl_flag(u + D);
      }
    }
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
    if (OVL && timed_out && lane == 0) atomicMax(a.status, kDevWaitTimeout);
  }

  if (a.s_final) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int e = 0; e < 4; ++e)
        a.s_final[sbase + (size_t)(row0 + 16 * i + 4 * grp + e) * DV + dv] = H[i][e];
  }
}

}  // namespace hagdn
