// k0_chunk_index.hip -- builds the chunk and segment tables of a packed
// (varlen) batch on the device, with no host synchronisation.
//
// Sequences are cut into chunks of 64 tokens that restart at every sequence
// start; the last chunk of a sequence may be partial.  Chunks are grouped into
// segments of seg_chunks chunks per sequence (the last may be shorter; an
// empty sequence gets one empty segment, so that every sequence has a
// workgroup that writes its final state).  The tables let the chunk-parallel
// kernels map blockIdx -> (sequence, first token, length) and the segment
// kernels walk one segment's chunks.  The kernel also checks the
// device-resident cu_seqlens (cu[0] = 0, nondecreasing, cu[N] = T); if they
// are malformed every sequence gets zero chunks and one empty segment (later
// kernels then touch no token and write the initial state as the final one)
// and it records HAGDN_DEV_BAD_SEQLENS.
//
// Bounds: sum_n ceil(len_n / 64) <= floor(T / 64) + N = max_chunks, and
// sum_n max(1, ceil(nch_n / L)) <= floor(max_chunks / L) + N = max_segs, so
// every index of a valid batch fits the tables the host sized.
#include "prefill.h"

namespace hagdn {

constexpr int kIndexThreads = 256;

__global__ __launch_bounds__(kIndexThreads) void chunk_index_kernel(PrefillArgs a) {
  const int tid = threadIdx.x;
  const int N = a.N;
  const int L = a.seg_chunks;
  const int32_t *cu = a.cu_seqlens;
  __shared__ int s_scan[2][kIndexThreads];
  __shared__ int s_carry[2];
  __shared__ int4 s_info[kIndexThreads];  // the first kIndexThreads sequences' tables
  __shared__ int2 s_seg[kIndexThreads];

  int bad = 0;
  int cu0 = 0, cu1 = 0;  // cu[tid], cu[tid + 1]: the first scan pass reuses them
  for (int n = tid; n < N; n += kIndexThreads) {
    const int x0 = cu[n], x1 = cu[n + 1];
    if (x1 < x0) bad = 1;
    if (n == tid) {
      cu0 = x0;
      cu1 = x1;
    }
  }
  if (tid == 0 && (cu[0] != 0 || cu[N] != a.T)) bad = 1;
  bad = __syncthreads_or(bad);

  if (tid < 2) s_carry[tid] = 0;
  __syncthreads();
  // exclusive scans of per-sequence chunk and segment counts, 256 sequences at a time
  for (int base = 0; base < N; base += kIndexThreads) {
    const int n = base + tid;
    int st = 0, len = 0;
    if (n < N && !bad) {
      st = base == 0 ? cu0 : cu[n];
      len = (base == 0 ? cu1 : cu[n + 1]) - st;
    }
    const int nch = (len + kChunk - 1) / kChunk;
    const int nseg = n < N ? max(1, (nch + L - 1) / L) : 0;
    s_scan[0][tid] = nch;
    s_scan[1][tid] = nseg;
    __syncthreads();
    for (int off = 1; off < kIndexThreads; off <<= 1) {
      const int add0 = tid >= off ? s_scan[0][tid - off] : 0;
      const int add1 = tid >= off ? s_scan[1][tid - off] : 0;
      __syncthreads();
      s_scan[0][tid] += add0;
      s_scan[1][tid] += add1;
      __syncthreads();
    }
    if (n < N) {
      const int4 si = make_int4(s_carry[0] + s_scan[0][tid] - nch, nch, st, len);
      const int2 ss = make_int2(s_carry[1] + s_scan[1][tid] - nseg, nseg);
      a.seq_info[n] = si;
      a.seq_seg[n] = ss;
      if (base == 0) {
        s_info[tid] = si;
        s_seg[tid] = ss;
      }
    }
    __syncthreads();
    if (tid == kIndexThreads - 1) {
      s_carry[0] += s_scan[0][tid];
      s_carry[1] += s_scan[1][tid];
    }
    __syncthreads();
  }
  int total = s_carry[0], total_segs = s_carry[1];
  // a batch of at most kIndexThreads sequences keeps its tables in LDS (one
  // scan pass): the chunk and segment loops below then search LDS instead of
  // reading the tables back from memory
  const bool lds_tables = N <= kIndexThreads;
  // cannot happen for a valid batch; keeps every later index in range anyway
  if (total > a.max_chunks || total_segs > a.max_segs) {
    bad = 1;
    total = 0;
    total_segs = N;  // <= max_segs
    for (int n = tid; n < N; n += kIndexThreads) {
      a.seq_info[n] = make_int4(0, 0, 0, 0);
      a.seq_seg[n] = make_int2(n, 1);
      if (n < kIndexThreads) {
        s_info[n] = make_int4(0, 0, 0, 0);
        s_seg[n] = make_int2(n, 1);
      }
    }
  }
  __threadfence_block();
  __syncthreads();

  for (int c = tid; c < a.max_chunks; c += kIndexThreads) {
    int4 info = make_int4(0, 0, 0, 0);
    if (!bad && c < total) {
      // last sequence whose first chunk is <= c (empty sequences share their
      // successor's first chunk and are skipped by taking the last match)
      int lo = 0, hi = N - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((lds_tables ? s_info[mid].x : a.seq_info[mid].x) <= c) lo = mid; else hi = mid - 1;
      }
      const int4 s = lds_tables ? s_info[lo] : a.seq_info[lo];
      const int j = c - s.x;
      if (j >= 0 && j < s.y) {
        const int off = j * kChunk;
        info = make_int4(lo, s.z + off, min(kChunk, s.w - off), 0);
      }
    }
    a.chunk_info[c] = info;
  }
  for (int sg = tid; sg < a.max_segs; sg += kIndexThreads) {
    int4 info = make_int4(-1, 0, 0, 0);
    if (sg < total_segs) {
      // every sequence has >= 1 segment, so first segments strictly increase
      int lo = 0, hi = N - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((lds_tables ? s_seg[mid].x : a.seq_seg[mid].x) <= sg) lo = mid; else hi = mid - 1;
      }
      const int2 ss = lds_tables ? s_seg[lo] : a.seq_seg[lo];
      const int j = sg - ss.x;
      if (j >= 0 && j < ss.y) {
        const int4 s = lds_tables ? s_info[lo] : a.seq_info[lo];
        info = make_int4(lo, s.x + j * L, min(L, s.y - j * L), j);
      }
    }
    a.seg_info[sg] = info;
  }
  if (tid == 0) a.status[0] = bad ? 1 : 0;
}

hipError_t launch_chunk_index(const PrefillArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL(chunk_index_kernel, dim3(1), dim3(kIndexThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace hagdn
