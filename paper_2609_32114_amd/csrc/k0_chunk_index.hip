// k0_chunk_index.hip -- builds the chunk table of a packed (varlen) batch on
// the device, with no host synchronisation.
//
// Sequences are cut into chunks of 64 tokens that restart at every sequence
// start; the last chunk of a sequence may be partial.  The table lets the
// chunk-parallel kernels map blockIdx -> (sequence, first token, length) and
// the sequential kernel walk one sequence's chunks.  It also checks the
// device-resident cu_seqlens (cu[0] = 0, nondecreasing, cu[N] = T); if they
// are malformed it writes an empty table (every later kernel then does no
// token work and stays in bounds) and records HAGDN_DEV_BAD_SEQLENS.
//
// Bound: sum_n ceil(len_n / 64) <= floor(T / 64) + N = max_chunks, so every
// chunk index of a valid batch fits the table the host sized.
#include "prefill.h"

namespace hagdn {

constexpr int kIndexThreads = 256;

__global__ __launch_bounds__(kIndexThreads) void chunk_index_kernel(PrefillArgs a) {
  const int tid = threadIdx.x;
  const int N = a.N;
  const int32_t *cu = a.cu_seqlens;
  __shared__ int s_scan[kIndexThreads];
  __shared__ int s_carry;

  int bad = 0;
  for (int n = tid; n < N; n += kIndexThreads)
    if (cu[n + 1] < cu[n]) bad = 1;
  if (tid == 0 && (cu[0] != 0 || cu[N] != a.T)) bad = 1;
  bad = __syncthreads_or(bad);

  if (tid == 0) s_carry = 0;
  __syncthreads();
  // exclusive scan of per-sequence chunk counts, 256 sequences at a time
  for (int base = 0; base < N; base += kIndexThreads) {
    const int n = base + tid;
    int st = 0, len = 0;
    if (n < N && !bad) {
      st = cu[n];
      len = cu[n + 1] - st;
    }
    const int nch = (len + kChunk - 1) / kChunk;
    s_scan[tid] = nch;
    __syncthreads();
    for (int off = 1; off < kIndexThreads; off <<= 1) {
      const int add = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += add;
      __syncthreads();
    }
    const int first = s_carry + s_scan[tid] - nch;
    if (n < N) a.seq_info[n] = make_int4(first, nch, st, len);
    __syncthreads();
    if (tid == kIndexThreads - 1) s_carry += s_scan[tid];
    __syncthreads();
  }
  const int total = s_carry;
  // cannot happen for a valid batch; keeps every later index in range anyway
  if (total > a.max_chunks) {
    bad = 1;
    for (int n = tid; n < N; n += kIndexThreads) a.seq_info[n] = make_int4(0, 0, 0, 0);
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
        if (a.seq_info[mid].x <= c) lo = mid; else hi = mid - 1;
      }
      const int4 s = a.seq_info[lo];
      const int j = c - s.x;
      if (j >= 0 && j < s.y) {
        const int off = j * kChunk;
        info = make_int4(lo, s.z + off, min(kChunk, s.w - off), 0);
      }
    }
    a.chunk_info[c] = info;
  }
  if (tid == 0) a.status[0] = bad ? 1 : 0;
}

hipError_t launch_chunk_index(const PrefillArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL(chunk_index_kernel, dim3(1), dim3(kIndexThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace hagdn
