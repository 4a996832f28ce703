/* Host-side checks of the C ABI (include/hagdn.h) for a sanitizer build:
 * every argument check, size computation, launch decision and error path that
 * runs on the host, with the kernel launchers stubbed out (stubs.cpp) so that
 * no GPU is needed.  Built with AddressSanitizer and UndefinedBehaviorSanitizer
 * on the host side by tests/test_host_sanitizers.py; any out-of-bounds access,
 * overflow or other undefined behaviour in the host code aborts the run.
 * Prints "host checks passed" and returns 0 when every expectation holds. */
#include <limits.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "hagdn.h"

static int failures = 0;

#define EXPECT(cond)                                                               \
  do {                                                                             \
    if (!(cond)) {                                                                 \
      fprintf(stderr, "line %d: expected %s (last error: %s)\n", __LINE__, #cond, \
              hagdn_last_error());                                                 \
      ++failures;                                                                  \
    }                                                                              \
  } while (0)

/* Device pointers are never dereferenced on the host: aligned stand-in addresses. */
#define FAKE(a) ((void *)(uintptr_t)(a))

static void sizes(void) {
  static const int Ns[] = {1, 2, 9, 1000};
  static const int Ts[] = {0, 1, 63, 64, 65, 4096, 32768, 1 << 20};
  static const int dims[] = {64, 128};
  for (int kda = 0; kda < 2; ++kda)
    for (size_t a = 0; a < sizeof Ns / sizeof *Ns; ++a)
      for (size_t b = 0; b < sizeof Ts / sizeof *Ts; ++b)
        for (int dk = 0; dk < 2; ++dk)
          for (int dv = 0; dv < 2; ++dv)
            for (int dt = 0; dt < 2; ++dt) {
              const int N = Ns[a], T = Ts[b];
              const size_t w = kda ? kda_prefill_workspace_size(N, T, 4, 16, dims[dk], dims[dv], dt)
                                   : gdn_prefill_workspace_size(N, T, 4, 16, dims[dk], dims[dv], dt);
              EXPECT(w > 0 && w % 256 == 0);
              for (int r = HAGDN_WS_NM; r <= HAGDN_WS_SEG_B; ++r) {
                size_t off = 0, bytes = 0;
                EXPECT(hagdn_workspace_region(kda, N, T, 4, 16, dims[dk], dims[dv], dt, r, &off, &bytes) ==
                       HAGDN_OK);
                EXPECT(off + bytes <= w);
              }
            }
  /* invalid shapes: 0 and a message */
  EXPECT(gdn_prefill_workspace_size(0, 10, 1, 1, 64, 64, HAGDN_F32) == 0 && hagdn_last_error()[0]);
  EXPECT(gdn_prefill_workspace_size(1, -1, 1, 1, 64, 64, HAGDN_F32) == 0);
  EXPECT(gdn_prefill_workspace_size(1, 10, 3, 4, 64, 64, HAGDN_F32) == 0);   /* Hv % Hqk */
  EXPECT(gdn_prefill_workspace_size(1, 10, 1, 1, 96, 64, HAGDN_F32) == 0);   /* Dk */
  EXPECT(gdn_prefill_workspace_size(1, 10, 1, 1, 64, 64, 7) == 0);          /* dtype */
  EXPECT(gdn_prefill_workspace_size(1, 10, 1, 70000, 64, 64, HAGDN_F32) == 0);
  /* sizes that would overflow are rejected, not wrapped */
  EXPECT(gdn_prefill_workspace_size(INT_MAX, INT_MAX, 65535, 65535, 128, 128, HAGDN_F32) == 0);
  EXPECT(kda_prefill_workspace_size(1, INT_MAX, 1, 65535, 128, 128, HAGDN_F32) > 0 ||
         hagdn_last_error()[0]);
  size_t off, bytes;
  EXPECT(hagdn_workspace_region(0, 1, 100, 1, 1, 64, 64, HAGDN_F32, 99, &off, &bytes) != HAGDN_OK);
}

static void rules(void) {
  for (int cus = 1; cus <= 512; cus += 37)
    for (int T = 0; T <= 1 << 18; T = T ? T * 3 : 1)
      for (int kda = 0; kda < 2; ++kda) {
        const int L = hagdn_segment_chunks_for(2, T, 16, 128, HAGDN_BF16, kda, cus);
        EXPECT(L >= 1);
        const int ov = hagdn_overlap_for(2, T, 16, 128, 128, HAGDN_BF16, kda, cus);
        EXPECT(ov == 0 || ov == 1);
      }
  EXPECT(hagdn_segment_chunks_for(1, 100, 16, 128, HAGDN_BF16, 0, 0) == -1);
  EXPECT(hagdn_overlap_for(1, 100, 16, 128, 128, HAGDN_BF16, 0, 0) == -1);
  EXPECT(hagdn_overlap_for(1, 4096, 16, 128, 128, HAGDN_BF16, 0, 256) == 1);
  EXPECT(hagdn_set_overlap(3) == HAGDN_EINVAL);
  EXPECT(hagdn_set_overlap(-1) == HAGDN_EINVAL);
  EXPECT(hagdn_overlap_for(1, 2048, 16, 128, 128, HAGDN_BF16, 0, 256) == 0);
  EXPECT(hagdn_set_overlap(2) == HAGDN_OK);
  EXPECT(hagdn_overlap_for(1, 2048, 16, 128, 128, HAGDN_BF16, 0, 256) == 1);
  EXPECT(hagdn_overlap_for(1, 2048, 16, 128, 128, HAGDN_BF16, 1, 256) == 0);
  EXPECT(hagdn_set_overlap(0) == HAGDN_OK);
  EXPECT(hagdn_overlap_for(1, 4096, 16, 128, 128, HAGDN_BF16, 0, 256) == 0);
  EXPECT(hagdn_set_overlap(1) == HAGDN_OK);
  EXPECT(hagdn_set_segment_chunks(-1) == HAGDN_EINVAL);
  EXPECT(hagdn_set_segment_chunks((1 << 20) + 1) == HAGDN_EINVAL);
  EXPECT(hagdn_set_segment_chunks(5) == HAGDN_OK);
  EXPECT(hagdn_segment_chunks(1, 100000, 16, 128, HAGDN_BF16, 0) == 5);
  EXPECT(hagdn_set_segment_chunks(0) == HAGDN_OK);
  EXPECT(hagdn_kernel_count() > 0);
  for (int i = -1; i <= hagdn_kernel_count(); ++i) EXPECT(hagdn_kernel_name(i) != NULL);
  EXPECT(hagdn_kernel_name(hagdn_kernel_count())[0] == 0);
  EXPECT(hagdn_version() > 0);
  EXPECT(hagdn_prefill_noalloc_capacity() > 0);
}

static void prefill_paths(void) {
  const int N = 2, T = 300, Hqk = 2, Hv = 4, D = 64;
  /* stand-ins 16 MiB apart, so that no two buffers overlap */
  int32_t *cu = FAKE(1ull << 24);
  void *q = FAKE(2ull << 24), *k = FAKE(3ull << 24), *v = FAKE(4ull << 24), *o = FAKE(5ull << 24);
  float *g = FAKE(6ull << 24), *b = FAKE(7ull << 24), *s0 = FAKE(8ull << 24), *sf = FAKE(9ull << 24);
  void *ws = FAKE(10ull << 24);
  const size_t wb = gdn_prefill_workspace_size(N, T, Hqk, Hv, D, D, HAGDN_BF16);
  EXPECT(wb > 0);
  /* argument checks, each before anything is enqueued */
  EXPECT(gdn_prefill(q, k, v, g, b, s0, NULL, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, o, sf, ws, wb, NULL) ==
         HAGDN_EINVAL);
  EXPECT(gdn_prefill(NULL, k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, o, sf, ws, wb, NULL) ==
         HAGDN_EINVAL);
  EXPECT(gdn_prefill(FAKE((2ull << 24) + 8), k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, o, sf, ws, wb,
                     NULL) == HAGDN_EINVAL); /* misaligned */
  EXPECT(gdn_prefill(q, k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, o, sf, ws, wb - 256, NULL) ==
         HAGDN_EWORKSPACE);
  EXPECT(gdn_prefill(q, k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, o, FAKE((8ull << 24) + 16), ws, wb,
                     NULL) == HAGDN_EINVAL); /* s_final overlaps s0 */
  EXPECT(gdn_prefill(q, k, v, g, b, s0, cu, N, T, Hqk, Hv, 96, D, 1.f, HAGDN_BF16, o, sf, ws, wb, NULL) ==
         HAGDN_EUNSUPPORTED);
  EXPECT(gdn_prefill_ex(q, k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, 8, o, sf, ws, wb, NULL) ==
         HAGDN_EINVAL); /* unknown flag */
  /* valid calls reach the (stubbed) launches: every path reports the HIP error */
  EXPECT(gdn_prefill(q, k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, o, sf, ws, wb, NULL) ==
         HAGDN_EHIP);
  EXPECT(kda_prefill_ex(q, k, v, g, b, NULL, cu, 1, 4096, 16, 16, 128, 128, 1.f, HAGDN_BF16, 7, o, NULL, ws,
                        kda_prefill_workspace_size(1, 4096, 16, 16, 128, 128, HAGDN_BF16), NULL) == HAGDN_EHIP);
  EXPECT(gdn_prefill(q, k, v, g, b, s0, cu, 1, 1 << 16, 16, 16, 128, 128, 1.f, HAGDN_BF16, o, s0, ws,
                     gdn_prefill_workspace_size(1, 1 << 16, 16, 16, 128, 128, HAGDN_BF16), NULL) == HAGDN_EHIP);
  /* an empty batch launches nothing that reads tokens (but still the tables) */
  EXPECT(gdn_prefill(NULL, NULL, NULL, NULL, NULL, NULL, cu, 1, 0, 1, 1, D, D, 1.f, HAGDN_F32, NULL, sf, ws,
                     gdn_prefill_workspace_size(1, 0, 1, 1, D, D, HAGDN_F32), NULL) != HAGDN_EINVAL);
  EXPECT(hagdn_prefill_noalloc(0, q, k, v, g, b, s0, cu, N, T, Hqk, Hv, D, D, 1.f, HAGDN_BF16, 0, o, sf, NULL) !=
         HAGDN_OK); /* no device to hold the array */
  EXPECT(hagdn_prefill_noalloc(0, q, k, v, g, b, s0, cu, 1, 1 << 24, 16, 16, 128, 128, 1.f, HAGDN_BF16, 0, o,
                               sf, NULL) == HAGDN_EWORKSPACE);
  int code = -1;
  EXPECT(hagdn_device_status(NULL, 0, NULL, &code) != HAGDN_OK);
}

static void decode_paths(void) {
  void *q = FAKE(0x20000), *k = FAKE(0x30000), *v = FAKE(0x40000), *o = FAKE(0x50000);
  float *g = FAKE(0x60000), *b = FAKE(0x70000), *st = FAKE(0x80000);
  int32_t *slots = FAKE(0x90000);
  EXPECT(gdn_decode(q, k, v, g, b, st, slots, 0, 4, 1, 1, 64, 64, 1.f, HAGDN_F32, 0, o, NULL) == HAGDN_EINVAL);
  EXPECT(gdn_decode(q, k, v, g, b, NULL, NULL, 0, 4, 1, 1, 64, 64, 1.f, HAGDN_F32, 0, o, NULL) == HAGDN_EINVAL);
  EXPECT(gdn_decode(q, k, v, g, b, st, NULL, 0, -1, 1, 1, 64, 64, 1.f, HAGDN_F32, 0, o, NULL) == HAGDN_EINVAL);
  EXPECT(gdn_decode(q, k, v, g, b, st, NULL, 0, 0, 1, 1, 64, 64, 1.f, HAGDN_F32, 0, o, NULL) == HAGDN_OK);
  EXPECT(kda_decode(q, k, v, g, b, st, slots, 16, 4, 2, 4, 128, 64, 1.f, HAGDN_BF16, 7, o, NULL) == HAGDN_EHIP);
}

static void profiling_and_aids(void) {
  double ms[16];
  int calls = 0;
  EXPECT(hagdn_profile_end(ms, 16, &calls) == HAGDN_EINVAL); /* not started */
  EXPECT(hagdn_profile_begin(0) == HAGDN_EINVAL);
  (void)hagdn_profile_begin(4); /* may fail without a device; must not leak or crash */
  (void)hagdn_profile_end(ms, 16, &calls);
  double flops = 0;
  EXPECT(hagdn_measure_copy(FAKE(0x1000), FAKE(0x2000), 17, NULL) == HAGDN_EINVAL);
  EXPECT(hagdn_measure_mfma(0, FAKE(0x1000), 4096, &flops, NULL) == HAGDN_EINVAL);
}

int main(void) {
  sizes();
  rules();
  prefill_paths();
  decode_paths();
  profiling_and_aids();
  if (failures) {
    fprintf(stderr, "%d host check(s) failed\n", failures);
    return 1;
  }
  printf("host checks passed\n");
  return 0;
}
