// api.cpp -- the C ABI of include/hagdn.h: host-side argument checks,
// workspace carving and the launches, all on the caller's stream.
//
// One call enqueues, in stream order:
//   K0 chunk index    (1 workgroup)                        sequence/chunk/segment tables,
//                                                          cu_seqlens check
//   K1 chunk-local    (max_chunks x Hv workgroups)         operators #1-#4
//   then either, when a sequence can span two segments (segment-parallel path),
//   K2 seg transfer   (max_segs x Hv x 2 workgroups)       segment maps of operator #5
//   K3 seg state      (max_segs x Hv workgroups)           operator #5 per segment, fused
//                                                          with operator #6
//   or, when every sequence is one segment,
//   K3 state prop     (N x Hv x Dv/16 workgroups)          operator #5 per chain, fused
//                                                          with operator #6
// The decode entry points enqueue one kernel (k4_decode.hip) and use no
// workspace.  No allocation, no synchronisation, no pointer retained after
// return.
#include <hip/hip_runtime.h>

#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <string>
#include <vector>

#include "../../include/hagdn.h"
#include "prefill.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

constexpr size_t kAlign = 256;
constexpr int kNumKernels = 7;
const char *const kKernelNames[kNumKernels] = {"chunk_index", "chunk_local", "seg_transfer", "state_prop",
                                               "decode",      "overlap_setup", "overlapped"};
constexpr int kDecodeKernel = 4;

// Chunks per segment of the state chain; 0 = chosen per call (seg_chunks).
std::atomic<int> g_seg_override{0};
// The overlapped launch (hagdn_set_overlap): 0 never, 1 where it pays (the
// default), 2 wherever it can run (overlap_applies).
std::atomic<int> g_overlap{1};
constexpr int kMaxSegChunks = 1 << 20;
// Compute units assumed by the size and segment-length queries when no HIP
// device can be queried (a host without a GPU: nothing can launch there, the
// answers only describe an MI355X).  Calls that launch always query.
constexpr int kNoDeviceCus = 256;

// Compute units of the current device, queried once per device (0 if the
// query fails).  Both the segment rule and the choice of walk kernel use it.
int current_device_cus() {
  constexpr int kMaxDevices = 64;
  static std::atomic<int> cache[kMaxDevices];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  int n = dev >= 0 && dev < kMaxDevices ? cache[dev].load(std::memory_order_relaxed) : 0;
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 0;
    if (dev >= 0 && dev < kMaxDevices) cache[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}
int query_cus() {
  const int n = current_device_cus();
  return n > 0 ? n : kNoDeviceCus;
}

// Segment length for a batch of N sequences over T tokens on a device of
// `cus` compute units.  A chain of n chunks walked whole costs n dependent
// steps; its workgroups (one per sequence, value head and 16-column tile)
// occupy N Hv Dv/16 CUs.  Cut into segments of L, it costs about L steps for
// the segment maps, n / L for the prefix and L for the walk, each step about
// three times as long (one head-resident workgroup moves a whole head's
// operands through one CU), on about (n / L) Hv workgroups.
//
// The thresholds come from sweeps of single sequences on an MI355X (256 CUs;
// d = 128, bf16, operator totals in us, whole chain against the best L):
//   GDN, 16 heads (128 walk workgroups, half the CUs): T = 6144 (96 chunks)
//     135 against 141 (L = 12); 7168 (112) 162 against 161 (L = 8); 8192
//     (128) 185 against 176 (L = 12); 9216 235 against 200; 12288 341
//     against 267.  Segments pay from about 120 chunks, and the best L puts
//     about one segment workgroup on every CU: L = n Hv / cus, at least 12.
//   GDN, 32 heads (256 walk workgroups, every CU): 192 chunks 484 against
//     480 (L = 24), 256 chunks 596 against 619 (L = 32): the whole walk holds
//     longer, so the threshold grows with the walks' share of the CUs,
//     r = walks / (cus / 2): 120 r + 48 (r - 1) chunks.
//   KDA, 16 heads: T = 4096 128 against 132 (L = 8); 6144 180 against 176
//     (L = 8); 8192 251 against 217.  Its per-channel gate adds 8 KiB per
//     token (d = 128) to the chunk-local kernel's input and pushes the walk's
//     operands out of the Infinity Cache sooner: KDA segments from 88 r +
//     48 (r - 1) chunks with L at least 8.
// Both scale with the CU count only through r and L = n Hv / cus; a device
// with fewer CUs (a partition) segments earlier and with longer segments.
//
// Whatever the choice (or override), L is capped so that the o rows of one
// segment, 64 L Hv Dv elements, span less than 2 GiB: the walk kernels address
// a segment's rows through one buffer resource with 32-bit signed byte
// offsets.  A call whose chains do not fit one capped segment takes the
// segmented path, whose windows then fit too.
int seg_chunks(int N, int T, int Hv, int Dv, size_t esz, bool kda, int cus) {
  const size_t seg_rows_bytes = (size_t)hagdn::kChunk * (size_t)Hv * (size_t)Dv * esz;
  const long cap = std::max<long>(1, (long)(((size_t)1 << 31) - 1) / (long)seg_rows_bytes);
  const int ov = g_seg_override.load(std::memory_order_relaxed);
  long L;
  if (ov > 0) {
    L = ov;
  } else {
    const long n_all = ((long)T + hagdn::kChunk - 1) / hagdn::kChunk;  // longest possible chain
    const long n_avg = ((long)T / (N > 0 ? N : 1) + hagdn::kChunk - 1) / hagdn::kChunk;
    const double walks = (double)(N > 0 ? N : 1) * Hv * std::max(1, Dv / 16);
    const long c = std::max(2, cus);
    const double r = std::max(1.0, walks / (double)(c / 2));
    const double threshold = (kda ? 88.0 : 120.0) * r + 48.0 * (r - 1.0);
    if ((double)n_avg < threshold) L = n_all > 0 ? std::min<long>(n_all, kMaxSegChunks) : 1;
    else L = std::max<long>(kda ? 8 : 12, (n_all * Hv + c - 1) / c);
  }
  return (int)std::min(L, cap);
}

// Chunks of a T-token sequence (64-bit: T + 63 overflows int near INT_MAX).
long chunks_of(int T) { return ((long)T + hagdn::kChunk - 1) / hagdn::kChunk; }

bool mul_ok(size_t a, size_t b, size_t *out) { return !__builtin_mul_overflow(a, b, out); }
bool add_ok(size_t a, size_t b, size_t *out) { return !__builtin_add_overflow(a, b, out); }

// Byte offsets of every workspace region (each 256-byte aligned).
struct Layout {
  size_t status, seq_info, chunk_info, NM, Bc, Qp, Ol, dec, seq_seg, seg_info, Aseg, Bseg, s0c, ovl, total;
  int max_chunks, seg_chunks, max_segs;
};

// Returns false (with the error set) if the sizes overflow.
bool make_layout(int N, int T, int Hv, int Dk, int Dv, size_t esz, bool kda, int cus, Layout *L) {
  const size_t mc = (size_t)(T / hagdn::kChunk) + (size_t)N;
  if (mc > 0x7fffffffu) {
    fail(HAGDN_EINVAL, "too many chunks (%zu)", mc);
    return false;
  }
  L->max_chunks = (int)mc;
  L->seg_chunks = seg_chunks(N, T, Hv, Dv, esz, kda, cus);
  const size_t ms = mc / (size_t)L->seg_chunks + (size_t)N;
  L->max_segs = (int)ms;  // <= mc
  size_t blocks, sblocks;  // (chunk, value head) and (segment, value head) blocks
  if (!mul_ok(mc, (size_t)Hv, &blocks) || !mul_ok(ms, (size_t)Hv, &sblocks)) {
    fail(HAGDN_EINVAL, "workspace size overflows");
    return false;
  }
  size_t off = 0;
  bool ok = true;
  auto region = [&](size_t elems_per_block, size_t bytes_per_elem, size_t nblocks) {
    size_t at = (off + kAlign - 1) / kAlign * kAlign;
    size_t b = 0;
    ok = ok && mul_ok(elems_per_block, bytes_per_elem, &b) && mul_ok(b, nblocks, &b) &&
         add_ok(at, b, &off);
    return at;
  };
  const size_t C = hagdn::kChunk;
  L->status = region(1, sizeof(int), 1);
  L->seq_info = region(1, sizeof(int4), (size_t)N);
  L->chunk_info = region(1, sizeof(int4), mc);
  L->NM = region((size_t)Dk * Dk, esz, blocks);
  L->Bc = region((size_t)Dv * Dk, esz, blocks);
  L->Qp = region(C * Dk, esz, blocks);
  L->Ol = region(C * Dv, esz, blocks);
  L->dec = region((size_t)Dk, sizeof(float), blocks);
  L->seq_seg = region(1, sizeof(int2), (size_t)N);
  L->seg_info = region(1, sizeof(int4), ms);
  // segment maps exist only when a sequence can span two segments
  const bool maps = chunks_of(T) > L->seg_chunks;
  L->Aseg = region((size_t)Dk * Dk, esz, maps ? sblocks : 0);
  L->Bseg = region((size_t)Dk * Dv, sizeof(float), maps ? sblocks : 0);
  L->s0c = region((size_t)Dk * Dv, sizeof(float), maps ? (size_t)N * (size_t)Hv : 0);
  // overlapped launch: per-XCD queues, then a ready flag per block
  L->ovl = region(1, sizeof(int), (size_t)hagdn::kOvlFlags + blocks);
  L->total = (off + kAlign - 1) / kAlign * kAlign;
  if (!ok) fail(HAGDN_EINVAL, "workspace size overflows");
  return ok;
}

int check_shapes(int N, int T, int Hqk, int Hv, int Dk, int Dv, int dtype) {
  if (N < 1) return fail(HAGDN_EINVAL, "N must be >= 1 (got %d)", N);
  if (T < 0) return fail(HAGDN_EINVAL, "T_total must be >= 0 (got %d)", T);
  if (Hqk < 1 || Hv < 1) return fail(HAGDN_EINVAL, "head counts must be >= 1 (Hqk=%d Hv=%d)", Hqk, Hv);
  if (Hv % Hqk != 0) return fail(HAGDN_EINVAL, "Hv (%d) must be a multiple of Hqk (%d)", Hv, Hqk);
  if (Hv > 65535) return fail(HAGDN_EUNSUPPORTED, "Hv > 65535 unsupported");
  if ((Dk != 64 && Dk != 128) || (Dv != 64 && Dv != 128))
    return fail(HAGDN_EUNSUPPORTED, "head dims must be 64 or 128 (Dk=%d Dv=%d)", Dk, Dv);
  if (dtype != HAGDN_F32 && dtype != HAGDN_BF16)
    return fail(HAGDN_EUNSUPPORTED, "dtype %d unsupported", dtype);
  return HAGDN_OK;
}

// Whether a call runs the chunk-local kernel and the whole-chain walks in one
// overlapped launch (k1_chunk_local.hip, launch_overlapped).  It needs chains
// walked whole by the four-wave walk (no segment maps), an instance for the
// operands (overlap_supported), a device of at least 8 XCDs x 32 CUs (XCC ids
// 0-7) and walks on at most half the CUs, so that the chunk-local work keeps
// most of the device.  In the automatic mode it also needs more chunk-local
// blocks than one round of the standalone kernel (3 per CU): the overlapped
// call costs about 20 us until the first chunk is ready plus the walk at
// ~0.88 us per chunk, against the standalone chunk-local kernel plus the walk
// at ~0.74 us per chunk, so it pays once the chunk-local kernel needs a second
// round.  Single sequences, d = 128, 256 CUs (us per call, overlapped against
// serialized, interleaved in one process): 4096 tokens x 16 heads (1040
// blocks) 88.9 / 92.3; 6144 x 16 (1552) 120.5 / 128.2; 2048 x 16 (528) 55.0 /
// 52.1; 4096 x 8 (520) 76.4 / 71.9.
bool overlap_applies(bool bf16, bool kda, int Dk, int Dv, bool maps, int N, int T, int Hv, int cus) {
  const int mode = g_overlap.load(std::memory_order_relaxed);
  if (mode == 0 || maps || !hagdn::overlap_supported(bf16, kda, Dk, Dv)) return false;
  if (cus < hagdn::kXcdCount * 32) return false;
  const long walks = (long)N * Hv * (Dv / 16);
  if (walks > cus / 2) return false;
  const long blocks = ((long)T / hagdn::kChunk + N) * Hv;  // chunk-local blocks (an upper bound)
  return mode == 2 || blocks > 3L * cus;
}

size_t workspace_size(bool kda, int N, int T, int Hqk, int Hv, int Dk, int Dv, int dtype) {
  if (check_shapes(N, T, Hqk, Hv, Dk, Dv, dtype) != HAGDN_OK) return 0;
  Layout L;
  if (!make_layout(N, T, Hv, Dk, Dv, dtype == HAGDN_BF16 ? 2 : 4, kda, query_cus(), &L)) return 0;
  return L.total;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p % a) == 0; }

// ------------------------------------------------------------------ profiling
struct Profile {
  bool on = false;
  int max_calls = 0;
  int calls = 0;
  std::vector<hipEvent_t> ev;      // [max_calls][kNumKernels + 1]; ev[i + 1] ends kernel i
  std::vector<unsigned char> ran;  // [max_calls][kNumKernels]: kernel i launched (else no end event)
};
thread_local Profile g_prof;

void prof_release() {
  for (hipEvent_t e : g_prof.ev) (void)hipEventDestroy(e);
  g_prof.ev.clear();
  g_prof.ran.clear();
  g_prof.on = false;
  g_prof.calls = g_prof.max_calls = 0;
}

int prefill(bool kda, const void *q, const void *k, const void *v, const float *g,
            const float *beta, const float *s0, const int32_t *cu, int N, int T, int Hqk, int Hv,
            int Dk, int Dv, float scale, int dtype, int pre, void *o, float *s_final, void *ws,
            size_t ws_bytes, void *stream_) {
  int rc = check_shapes(N, T, Hqk, Hv, Dk, Dv, dtype);
  if (rc != HAGDN_OK) return rc;
  if (pre & ~hagdn::kPreAll) return fail(HAGDN_EINVAL, "unknown preprocessing flags 0x%x", pre);
  if (!cu || !ws) return fail(HAGDN_EINVAL, "NULL required pointer (cu_seqlens, workspace)");
  // token tensors are never dereferenced for an empty batch (torch hands out
  // NULL for zero-size allocations)
  if (T > 0 && (!q || !k || !v || !g || !beta || !o))
    return fail(HAGDN_EINVAL, "NULL required pointer (q, k, v, g, beta, o)");
  const void *p16[] = {q, k, v, o, s0, s_final, ws};
  const char *n16[] = {"q", "k", "v", "o", "s0", "s_final", "workspace"};
  for (int i = 0; i < 7; ++i)
    if (p16[i] && !aligned(p16[i], 16)) return fail(HAGDN_EINVAL, "%s is not 16-byte aligned", n16[i]);
  if (!aligned(g, 4) || !aligned(beta, 4) || !aligned(cu, 4))
    return fail(HAGDN_EINVAL, "g, beta and cu_seqlens must be 4-byte aligned");
  if (s_final && s0 && s_final != s0) {
    const size_t sb = (size_t)N * Hv * Dk * Dv * sizeof(float);
    const char *a0 = (const char *)s0, *a1 = (const char *)s_final;
    if (a0 < a1 + sb && a1 < a0 + sb) return fail(HAGDN_EINVAL, "s_final overlaps s0 without aliasing it exactly");
  }
  const bool bf16 = dtype == HAGDN_BF16;
  const int cus = query_cus();  // the workspace-size query's answer for this device
  Layout L;
  if (!make_layout(N, T, Hv, Dk, Dv, bf16 ? 2 : 4, kda, cus, &L)) return HAGDN_EINVAL;
  if (ws_bytes < L.total)
    return fail(HAGDN_EWORKSPACE, "workspace too small: %zu bytes given, %zu needed", ws_bytes, L.total);

  char *w = static_cast<char *>(ws);
  hagdn::PrefillArgs a;
  a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta; a.s0 = s0; a.cu_seqlens = cu;
  a.N = N; a.T = T; a.Hqk = Hqk; a.Hv = Hv; a.Dk = Dk; a.Dv = Dv;
  a.max_chunks = L.max_chunks;
  a.scale = scale;
  a.pre = pre;
  a.o = o; a.s_final = s_final;
  a.status = reinterpret_cast<int *>(w + L.status);
  a.seq_info = reinterpret_cast<int4 *>(w + L.seq_info);
  a.chunk_info = reinterpret_cast<int4 *>(w + L.chunk_info);
  a.NM = w + L.NM; a.Bc = w + L.Bc; a.Qp = w + L.Qp; a.Ol = w + L.Ol;
  a.dec = reinterpret_cast<float *>(w + L.dec);
  a.seg_chunks = L.seg_chunks;
  a.max_segs = L.max_segs;
  a.seq_seg = reinterpret_cast<int2 *>(w + L.seq_seg);
  a.seg_info = reinterpret_cast<int4 *>(w + L.seg_info);
  a.Aseg = w + L.Aseg;
  a.Bseg = reinterpret_cast<float *>(w + L.Bseg);
  a.s0c = reinterpret_cast<float *>(w + L.s0c);
  a.single = N == 1 ? 1 : 0;  // the kernels derive a single sequence's tables themselves
  a.cus = cus;
  a.ovl = reinterpret_cast<int *>(w + L.ovl);
  a.ovl_walk_wgs = 0;
  const bool maps = chunks_of(T) > L.seg_chunks;
  const bool overlap = T > 0 && overlap_applies(bf16, kda, Dk, Dv, maps, N, T, Hv, cus);

  hipStream_t st = static_cast<hipStream_t>(stream_);
  hipEvent_t *ev = nullptr;
  unsigned char *ran = nullptr;
  if (g_prof.on && g_prof.calls < g_prof.max_calls) {
    ev = &g_prof.ev[(size_t)g_prof.calls * (kNumKernels + 1)];
    ran = &g_prof.ran[(size_t)g_prof.calls * kNumKernels];
    ++g_prof.calls;
    for (int i = 0; i < kNumKernels; ++i) ran[i] = 0;
  }
  // mark(i): event i (i = 0: before the first kernel; i > 0: kernel i-1 ended)
  auto mark = [&](int i) -> hipError_t {
    if (!ev) return hipSuccess;
    if (i > 0) ran[i - 1] = 1;
    return hipEventRecord(ev[i], st);
  };

  hipError_t e;
  if ((e = mark(0)) != hipSuccess) goto hip_fail;
  if (!a.single) {
    if ((e = hagdn::launch_chunk_index(a, st)) != hipSuccess) goto hip_fail;
    if ((e = mark(1)) != hipSuccess) goto hip_fail;
  }
  if (overlap) {
    // flags and queues cleared (and a single sequence's status word written),
    // then the chunk-local items and the walks in one launch
    if ((e = hagdn::launch_overlap_setup(a, st)) != hipSuccess) goto hip_fail;
    if ((e = mark(6)) != hipSuccess) goto hip_fail;
    if ((e = hagdn::launch_overlapped(a, st)) != hipSuccess) goto hip_fail;
    if ((e = mark(7)) != hipSuccess) goto hip_fail;
    return HAGDN_OK;
  }
  if ((e = hagdn::launch_chunk_local(a, bf16, kda, st)) != hipSuccess) goto hip_fail;
  if ((e = mark(2)) != hipSuccess) goto hip_fail;
  if (maps) {
    if ((e = hagdn::launch_seg_transfer(a, bf16, kda, st)) != hipSuccess) goto hip_fail;
    if ((e = mark(3)) != hipSuccess) goto hip_fail;
  }
  if ((e = maps ? hagdn::launch_seg_state(a, bf16, kda, st) : hagdn::launch_state_prop(a, bf16, kda, st)) !=
      hipSuccess)
    goto hip_fail;
  if ((e = mark(4)) != hipSuccess) goto hip_fail;
  return HAGDN_OK;
hip_fail:
  return fail(HAGDN_EHIP, "HIP error: %s", hipGetErrorString(e));
}

int decode(bool kda, const void *q, const void *k, const void *v, const float *g,
           const float *beta, float *state, const int32_t *slots, int num_slots, int N, int Hqk,
           int Hv, int Dk, int Dv, float scale, int dtype, int pre, void *o, void *stream) {
  if (N < 0) return fail(HAGDN_EINVAL, "N must be >= 0 (got %d)", N);
  int rc = check_shapes(N > 0 ? N : 1, 0, Hqk, Hv, Dk, Dv, dtype);
  if (rc != HAGDN_OK) return rc;
  if (pre & ~hagdn::kPreAll) return fail(HAGDN_EINVAL, "unknown preprocessing flags 0x%x", pre);
  if (N == 0) return HAGDN_OK;
  if (!slots) num_slots = N;
  if (num_slots < 1) return fail(HAGDN_EINVAL, "num_slots must be >= 1 (got %d)", num_slots);
  if ((size_t)N * Hv * (Dv / 64) > 0x7fffffffu) return fail(HAGDN_EINVAL, "N x Hv too large");
  if (!q || !k || !v || !g || !beta || !state || !o)
    return fail(HAGDN_EINVAL, "NULL required pointer (q, k, v, g, beta, state, o)");
  const void *p16[] = {q, k, v, o, state};
  const char *n16[] = {"q", "k", "v", "o", "state"};
  for (int i = 0; i < 5; ++i)
    if (!aligned(p16[i], 16)) return fail(HAGDN_EINVAL, "%s is not 16-byte aligned", n16[i]);
  if (!aligned(g, 4) || !aligned(beta, 4) || !aligned(slots, 4))
    return fail(HAGDN_EINVAL, "g, beta and slots must be 4-byte aligned");
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipEvent_t *ev = nullptr;
  if (g_prof.on && g_prof.calls < g_prof.max_calls) {
    ev = &g_prof.ev[(size_t)g_prof.calls * (kNumKernels + 1)];
    unsigned char *ran = &g_prof.ran[(size_t)g_prof.calls * kNumKernels];
    ++g_prof.calls;
    for (int i = 0; i < kNumKernels; ++i) ran[i] = i == kDecodeKernel;
  }
  hagdn::DecodeArgs a;
  a.q = q; a.k = k; a.v = v; a.g = g; a.beta = beta; a.state = state; a.slots = slots;
  a.N = N; a.Hqk = Hqk; a.Hv = Hv; a.Dk = Dk; a.Dv = Dv; a.num_slots = num_slots;
  a.scale = scale; a.pre = pre; a.o = o;
  hipError_t e = ev ? hipEventRecord(ev[0], st) : hipSuccess;
  if (e == hipSuccess) e = hagdn::launch_decode(a, dtype == HAGDN_BF16, kda, st);
  if (e == hipSuccess && ev) e = hipEventRecord(ev[kDecodeKernel + 1], st);
  if (e != hipSuccess) return fail(HAGDN_EHIP, "HIP error: %s", hipGetErrorString(e));
  return HAGDN_OK;
}

// ------------------------------------------------- allocation-free entry point
// The workspace of hagdn_prefill_noalloc: a file-scope device array, one copy
// per device, held until the process ends.  Host code must never pass the
// array's name to a kernel or a copy (it names a host-side stand-in); it uses
// the device address hipGetSymbolAddress returns, looked up once per device
// with that device current.
constexpr size_t kScratchBytes = (size_t)128 << 20;
__device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::atomic<void *> g_scratch_ptr[kMaxScratchDevices];

// Device address of `scratch` on the current device (looked up on first use).
hipError_t scratch_address(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  void *p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev].store(p, std::memory_order_release);  // the same address from any thread
  }
  *out = p;
  return hipSuccess;
}

}  // namespace

extern "C" {

int hagdn_prefill_noalloc(int kda, const void *q, const void *k, const void *v, const float *g,
                          const float *beta, const float *s0, const int32_t *cu_seqlens, int N,
                          int T_total, int Hqk, int Hv, int Dk, int Dv, float scale, int dtype,
                          int pre, void *o, float *s_final, void *stream) {
  int rc = check_shapes(N, T_total, Hqk, Hv, Dk, Dv, dtype);
  if (rc != HAGDN_OK) return rc;
  Layout L;
  if (!make_layout(N, T_total, Hv, Dk, Dv, dtype == HAGDN_BF16 ? 2 : 4, kda != 0, query_cus(), &L))
    return HAGDN_EINVAL;
  if (L.total > kScratchBytes)
    return fail(HAGDN_EWORKSPACE, "the call needs %zu bytes of workspace; hagdn_prefill_noalloc holds %zu",
                L.total, kScratchBytes);
  void *ws = nullptr;
  hipError_t e = scratch_address(&ws);
  if (e != hipSuccess) return fail(HAGDN_EHIP, "static workspace: %s", hipGetErrorString(e));
  return prefill(kda != 0, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv, Dk, Dv, scale, dtype,
                 pre, o, s_final, ws, kScratchBytes, stream);
}

size_t hagdn_prefill_noalloc_capacity(void) { return kScratchBytes; }

size_t gdn_prefill_workspace_size(int N, int T_total, int Hqk, int Hv, int Dk, int Dv, int dtype) {
  return workspace_size(false, N, T_total, Hqk, Hv, Dk, Dv, dtype);
}

size_t kda_prefill_workspace_size(int N, int T_total, int Hqk, int Hv, int Dk, int Dv, int dtype) {
  return workspace_size(true, N, T_total, Hqk, Hv, Dk, Dv, dtype);
}

int gdn_prefill(const void *q, const void *k, const void *v, const float *g, const float *beta,
                const float *s0, const int32_t *cu_seqlens, int N, int T_total, int Hqk, int Hv,
                int Dk, int Dv, float scale, int dtype, void *o, float *s_final, void *workspace,
                size_t workspace_bytes, void *stream) {
  return prefill(false, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv, Dk, Dv, scale,
                 dtype, 0, o, s_final, workspace, workspace_bytes, stream);
}

int gdn_prefill_ex(const void *q, const void *k, const void *v, const float *g, const float *beta,
                   const float *s0, const int32_t *cu_seqlens, int N, int T_total, int Hqk, int Hv,
                   int Dk, int Dv, float scale, int dtype, int pre, void *o, float *s_final,
                   void *workspace, size_t workspace_bytes, void *stream) {
  return prefill(false, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv, Dk, Dv, scale,
                 dtype, pre, o, s_final, workspace, workspace_bytes, stream);
}

int kda_prefill_ex(const void *q, const void *k, const void *v, const float *g, const float *beta,
                   const float *s0, const int32_t *cu_seqlens, int N, int T_total, int Hqk, int Hv,
                   int Dk, int Dv, float scale, int dtype, int pre, void *o, float *s_final,
                   void *workspace, size_t workspace_bytes, void *stream) {
  return prefill(true, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv, Dk, Dv, scale,
                 dtype, pre, o, s_final, workspace, workspace_bytes, stream);
}

int gdn_decode(const void *q, const void *k, const void *v, const float *g, const float *beta,
               float *state, const int32_t *slots, int num_slots, int N, int Hqk, int Hv, int Dk,
               int Dv, float scale, int dtype, int pre, void *o, void *stream) {
  return decode(false, q, k, v, g, beta, state, slots, num_slots, N, Hqk, Hv, Dk, Dv, scale, dtype,
                pre, o, stream);
}

int kda_decode(const void *q, const void *k, const void *v, const float *g, const float *beta,
               float *state, const int32_t *slots, int num_slots, int N, int Hqk, int Hv, int Dk,
               int Dv, float scale, int dtype, int pre, void *o, void *stream) {
  return decode(true, q, k, v, g, beta, state, slots, num_slots, N, Hqk, Hv, Dk, Dv, scale, dtype,
                pre, o, stream);
}

int kda_prefill(const void *q, const void *k, const void *v, const float *g, const float *beta,
                const float *s0, const int32_t *cu_seqlens, int N, int T_total, int Hqk, int Hv,
                int Dk, int Dv, float scale, int dtype, void *o, float *s_final, void *workspace,
                size_t workspace_bytes, void *stream) {
  return prefill(true, q, k, v, g, beta, s0, cu_seqlens, N, T_total, Hqk, Hv, Dk, Dv, scale,
                 dtype, 0, o, s_final, workspace, workspace_bytes, stream);
}

const char *hagdn_last_error(void) { return g_err.c_str(); }

int hagdn_device_status(const void *workspace, size_t workspace_bytes, void *stream, int *code) {
  if (!workspace || !code) return fail(HAGDN_EINVAL, "NULL workspace or code");
  if (workspace_bytes < sizeof(int)) return fail(HAGDN_EINVAL, "workspace too small");
  int host = -1;
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(&host, workspace, sizeof(int), hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return fail(HAGDN_EHIP, "HIP error: %s", hipGetErrorString(e));
  *code = host;
  return HAGDN_OK;
}

int hagdn_profile_begin(int max_calls) {
  if (max_calls < 1 || max_calls > (1 << 20)) return fail(HAGDN_EINVAL, "max_calls out of range");
  prof_release();
  g_prof.ev.assign((size_t)max_calls * (kNumKernels + 1), nullptr);
  g_prof.ran.assign((size_t)max_calls * kNumKernels, 0);
  for (hipEvent_t &e : g_prof.ev) {
    hipError_t r = hipEventCreate(&e);
    if (r != hipSuccess) {
      prof_release();
      return fail(HAGDN_EHIP, "hipEventCreate: %s", hipGetErrorString(r));
    }
  }
  g_prof.max_calls = max_calls;
  g_prof.calls = 0;
  g_prof.on = true;
  return HAGDN_OK;
}

int hagdn_profile_end(double *mean_ms, int max_kernels, int *calls) {
  if (!g_prof.on) return fail(HAGDN_EINVAL, "profiling was not started");
  const int nc = g_prof.calls;
  std::vector<double> sum(kNumKernels, 0.0);
  std::vector<int> runs(kNumKernels, 0);
  for (int c = 0; c < nc; ++c) {
    hipEvent_t *ev = &g_prof.ev[(size_t)c * (kNumKernels + 1)];
    const unsigned char *ran = &g_prof.ran[(size_t)c * kNumKernels];
    int last = -1;  // the call's last kernel: its end event is the call's last event
    for (int i = 0; i < kNumKernels; ++i)
      if (ran[i]) last = i;
    hipError_t r = last >= 0 ? hipEventSynchronize(ev[last + 1]) : hipSuccess;
    hipEvent_t prev = ev[0];
    for (int i = 0; i < kNumKernels && r == hipSuccess; ++i) {
      if (!ran[i]) continue;  // not launched in this call
      float ms = 0.f;
      r = hipEventElapsedTime(&ms, prev, ev[i + 1]);
      sum[i] += ms;
      ++runs[i];
      prev = ev[i + 1];
    }
    if (r != hipSuccess) {
      prof_release();
      return fail(HAGDN_EHIP, "event timing: %s", hipGetErrorString(r));
    }
  }
  for (int i = 0; i < kNumKernels && i < max_kernels && mean_ms; ++i)
    mean_ms[i] = runs[i] ? sum[i] / runs[i] : 0.0;
  if (calls) *calls = nc;
  prof_release();
  return HAGDN_OK;
}

int hagdn_kernel_count(void) { return kNumKernels; }

const char *hagdn_kernel_name(int i) { return (i >= 0 && i < kNumKernels) ? kKernelNames[i] : ""; }

int hagdn_version(void) { return 100; }

int hagdn_set_overlap(int mode) {
  if (mode < 0 || mode > 2) return fail(HAGDN_EINVAL, "overlap mode must be 0, 1 or 2 (got %d)", mode);
  g_overlap.store(mode, std::memory_order_relaxed);
  return HAGDN_OK;
}

int hagdn_overlap_for(int N, int T_total, int Hv, int Dk, int Dv, int dtype, int kda, int cus) {
  if (check_shapes(N, T_total, 1, Hv, Dk, Dv, dtype) != HAGDN_OK) return -1;
  if (cus < 1) return fail(HAGDN_EINVAL, "cus must be >= 1 (got %d)", cus), -1;
  const size_t esz = dtype == HAGDN_BF16 ? 2 : 4;
  const int L = seg_chunks(N, T_total, Hv, Dv, esz, kda != 0, cus);
  const bool maps = chunks_of(T_total) > L;
  return T_total > 0 && overlap_applies(dtype == HAGDN_BF16, kda != 0, Dk, Dv, maps, N, T_total, Hv, cus) ? 1 : 0;
}

int hagdn_set_segment_chunks(int chunks) {
  if (chunks < 0 || chunks > kMaxSegChunks)
    return fail(HAGDN_EINVAL, "segment length %d out of range [0, %d]", chunks, kMaxSegChunks);
  g_seg_override.store(chunks, std::memory_order_relaxed);
  return HAGDN_OK;
}

int hagdn_measure_copy(const void *src, void *dst, size_t bytes, void *stream) {
  if (!src || !dst) return fail(HAGDN_EINVAL, "NULL src or dst");
  if (bytes % 16 || !aligned(src, 16) || !aligned(dst, 16))
    return fail(HAGDN_EINVAL, "copy needs 16-byte aligned buffers and a multiple of 16 bytes");
  const char *a = static_cast<const char *>(src), *b = static_cast<const char *>(dst);
  if (a < b + bytes && b < a + bytes) return fail(HAGDN_EINVAL, "src and dst overlap");
  if (bytes == 0) return HAGDN_OK;
  hipError_t e = hagdn::launch_copy(src, dst, bytes, current_device_cus(), static_cast<hipStream_t>(stream));
  return e == hipSuccess ? HAGDN_OK : fail(HAGDN_EHIP, "HIP error: %s", hipGetErrorString(e));
}

int hagdn_measure_mfma(int iterations, float *sink, size_t sink_floats, double *flops, void *stream) {
  if (!sink || !flops) return fail(HAGDN_EINVAL, "NULL sink or flops");
  if (iterations < 1 || iterations > (1 << 24)) return fail(HAGDN_EINVAL, "iterations out of range [1, 2^24]");
  const int cus = current_device_cus();
  if (cus <= 0) return fail(HAGDN_EHIP, "cannot query the current HIP device");
  const int blocks = 4 * cus;  // four waves per workgroup: 16 waves per CU, 4 per SIMD
  if (sink_floats < (size_t)blocks * 4)
    return fail(HAGDN_EINVAL, "sink needs %d floats (4 per workgroup of 4 x CUs)", blocks * 4);
  if (!aligned(sink, 4)) return fail(HAGDN_EINVAL, "sink must be 4-byte aligned");
  hipError_t e = hagdn::launch_mfma_loop(blocks, iterations, sink, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(HAGDN_EHIP, "HIP error: %s", hipGetErrorString(e));
  *flops = 2.0 * 16 * 16 * 32 * 8 * (double)iterations * blocks * 4;
  return HAGDN_OK;
}

int hagdn_workspace_region(int kda, int N, int T_total, int Hqk, int Hv, int Dk, int Dv, int dtype,
                           int region, size_t *offset, size_t *bytes) {
  if (!offset || !bytes) return fail(HAGDN_EINVAL, "NULL offset or bytes");
  int rc = check_shapes(N, T_total, Hqk, Hv, Dk, Dv, dtype);
  if (rc != HAGDN_OK) return rc;
  Layout L;
  if (!make_layout(N, T_total, Hv, Dk, Dv, dtype == HAGDN_BF16 ? 2 : 4, kda != 0, query_cus(), &L))
    return HAGDN_EINVAL;
  size_t at, next;
  switch (region) {
    case HAGDN_WS_NM: at = L.NM; next = L.Bc; break;
    case HAGDN_WS_B: at = L.Bc; next = L.Qp; break;
    case HAGDN_WS_QP: at = L.Qp; next = L.Ol; break;
    case HAGDN_WS_OLOC: at = L.Ol; next = L.dec; break;
    case HAGDN_WS_DECAY: at = L.dec; next = L.seq_seg; break;
    case HAGDN_WS_SEG_A: at = L.Aseg; next = L.Bseg; break;
    case HAGDN_WS_SEG_B: at = L.Bseg; next = L.s0c; break;
    default: return fail(HAGDN_EINVAL, "unknown workspace region %d", region);
  }
  *offset = at;
  *bytes = next - at;  // the region plus its alignment padding
  return HAGDN_OK;
}

int hagdn_segment_chunks_for(int N, int T_total, int Hv, int Dv, int dtype, int kda, int cus) {
  if (N < 1 || T_total < 0 || Hv < 1 || Dv < 1)
    return fail(HAGDN_EINVAL, "bad shape"), -1;
  if (dtype != HAGDN_F32 && dtype != HAGDN_BF16) return fail(HAGDN_EINVAL, "bad dtype %d", dtype), -1;
  if (cus < 1) return fail(HAGDN_EINVAL, "compute units must be >= 1 (got %d)", cus), -1;
  return seg_chunks(N, T_total, Hv, Dv, dtype == HAGDN_BF16 ? 2 : 4, kda != 0, cus);
}

int hagdn_segment_chunks(int N, int T_total, int Hv, int Dv, int dtype, int kda) {
  return hagdn_segment_chunks_for(N, T_total, Hv, Dv, dtype, kda, query_cus());
}

}  // extern "C"
