/*
 * Host-side fuzz of the C ABI, built with AddressSanitizer and
 * UndefinedBehaviorSanitizer around the library's host code (abi.hip).
 *
 * Every entry point is called many times with arguments drawn from small
 * sets of edge values: NULL, aligned and misaligned stand-in device
 * addresses, negative, zero, tiny, large and overflowing sizes, unknown
 * dtype and activation codes.  Host pointers (counts the library writes
 * on the host) are real host variables.  On a machine without a GPU a call
 * that passes validation fails at its first HIP call, so no stand-in
 * address is ever dereferenced; the program refuses to run where a GPU is
 * present.  Every call must return a status code of the ABI and leave a
 * bounded, terminated message; the sanitizers abort on anything else.
 */
#include <limits.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "shc.h"

static uint64_t g_state = 0x2545F4914F6CDD1DULL;
static uint64_t next_u64(void) { /* splitmix64 */
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ULL);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}
#define PICK(arr) (arr[next_u64() % (sizeof(arr) / sizeof(arr[0]))])

static void* const kPtrs[] = {NULL, (void*)(uintptr_t)0x10000, (void*)(uintptr_t)0x10004,
                              (void*)(uintptr_t)0x7f0000001000ULL};
static const int64_t kI64[] = {-7, -1, 0, 1, 3, 16, 37, 655, 4097, 10475, 1 << 20,
                               INT32_MAX, (int64_t)INT32_MAX + 1, INT64_MAX / 2};
static const int32_t kI32[] = {-1, 0, 1, 2, 3, 9, 10, 16, 31, 32, 33, 48, 64, 128, 256,
                               257, 4096, 4112, 19456, 19457, INT32_MAX};
static const int32_t kCode[] = {-1, 0, 1, 2, 3};
static const size_t kSize[] = {0, 15, 256, 4096, (size_t)1 << 30, SIZE_MAX};
static const float kF[] = {0.0f, 1e-5f, -1.0f, 1e30f};

#define P() PICK(kPtrs)
#define I64() PICK(kI64)
#define I32() PICK(kI32)
#define CODE() PICK(kCode)
#define SZ() PICK(kSize)

static long g_calls = 0, g_ok = 0;
static int g_bad = 0;

static void check(int rc, const char* fn) {
  ++g_calls;
  if (rc == 0) ++g_ok;
  if (rc > 0 || rc < -5) {
    fprintf(stderr, "%s returned %d, not a status code\n", fn, rc);
    g_bad = 1;
  }
  const char* e = shc_last_error();
  if (e == NULL || strnlen(e, 1024) >= 512) {
    fprintf(stderr, "%s left an unterminated or overlong message\n", fn);
    g_bad = 1;
  }
  const char* st = shc_status_string(rc);
  if (st == NULL || strncmp(st, "SHC_", 4) != 0) {
    fprintf(stderr, "no status string for %d\n", rc);
    g_bad = 1;
  }
}

int main(void) {
  int ndev = 0;
  if (hipGetDeviceCount(&ndev) == hipSuccess && ndev > 0) {
    fprintf(stderr, "a GPU is present: this fuzz is for machines without one\n");
    return 2;
  }
  int64_t host_count = 0;
  int32_t kt_host = 0;
  void* ev = NULL;
  const int reps = 4000;
  for (int r = 0; r < reps; ++r) {
    (void)shc_compact_mask_workspace(I32(), I32());
    (void)shc_mask_scores_workspace(I32(), I64(), I32());
    (void)shc_transpose_neighbors_workspace(I32(), I32());
    (void)shc_sparse_linear_backward_workspace(I64(), I32(), I32(), CODE());
    (void)shc_build_slot_pairs_workspace(I64(), I32());
    (void)shc_sparse_neighbor_conv_backward_workspace(I64(), I32(), I32(), I32(), CODE());
    (void)shc_conv_plan_max_rows(I32(), I32(), I32(), CODE());
    (void)shc_conv_plan_bytes(I64(), I32(), I32(), I32(), CODE());
    host_count = (next_u64() & 1) ? -1 : 5;
    int64_t* hc = (next_u64() & 1) ? &host_count : NULL;
    check(shc_compact_mask(P(), I32(), I32(), P(), P(), P(), P(), hc, I64(), P(), SZ(), NULL),
          "compact_mask");
    check(shc_compact_mask_noalloc(P(), I32(), I32(), P(), P(), P(), P(), hc, I64(), NULL),
          "compact_mask_noalloc");
    check(shc_compact_mask_start(P(), I32(), I32(), P(), P(), P(), P(), hc, I64(), P(), SZ(),
                                 NULL),
          "compact_mask_start");
    host_count = 5;
    check(shc_compact_mask_wait((next_u64() & 1) ? &host_count : NULL, I64(), NULL),
          "compact_mask_wait");
    check(shc_compact_mask_table_start(P(), I32(), I32(), P(), P(), P(), P(), hc, I64(), P(),
                                       I32(), P(), P(), SZ(), NULL),
          "compact_mask_table_start");
    check(shc_gather_rows(P(), P(), I64(), I32(), I32(), I32(), CODE(), P(), NULL), "gather_rows");
    check(shc_gather_rows_stacked(P(), P(), I64(), I32(), I32(), I32(), I32(), CODE(), P(), NULL),
          "gather_rows_stacked");
    check(shc_combine_stacked(P(), I32(), I64(), I32(), CODE(), CODE(), P(), NULL),
          "combine_stacked");
    check(shc_row_mask_from_elements(P(), I32(), I32(), I32(), P(), NULL), "row_mask_from_elements");
    check(shc_gather_rows_masked(P(), P(), P(), I64(), I32(), I32(), I32(), CODE(), P(), NULL),
          "gather_rows_masked");
    check(shc_sparse_linear(P(), I64(), P(), P(), I32(), I32(), CODE(), CODE(), P(), NULL),
          "sparse_linear");
    check(shc_gather_sparse_linear(P(), P(), I64(), I32(), I32(), P(), P(), I32(), I32(), CODE(),
                                   CODE(), P(), NULL),
          "gather_sparse_linear");
    check(shc_sparse_neighbor_conv(P(), P(), P(), I64(), I32(), I32(), P(), I32(), P(), P(), I32(),
                                   I32(), CODE(), CODE(), P(), NULL),
          "sparse_neighbor_conv");
    check(shc_build_neighbor_table(P(), P(), I64(), I32(), I32(), P(), I32(), P(), NULL),
          "build_neighbor_table");
    check(shc_sparse_neighbor_conv_table(P(), P(), I64(), I32(), P(), P(), I32(), I32(), CODE(),
                                         CODE(), P(), NULL),
          "sparse_neighbor_conv_table");
    check(shc_build_conv_plan(P(), I64(), I32(), I32(), I32(), CODE(), P(), SZ(), NULL),
          "build_conv_plan");
    check(shc_sparse_neighbor_conv_planned(P(), P(), SZ(), I64(), I32(), P(), P(), I32(), I32(),
                                           CODE(), CODE(), P(), NULL),
          "sparse_neighbor_conv_planned");
    check(shc_scatter(P(), P(), P(), I64(), I32(), I32(), I32(), CODE(), CODE(), P(), NULL),
          "scatter");
    check(shc_clear_inactive_rows(P(), I32(), I32(), I32(), CODE(), P(), NULL),
          "clear_inactive_rows");
    check(shc_segment_group_norm(P(), P(), I64(), I32(), I32(), I32(), PICK(kF), CODE(), P(), NULL),
          "segment_group_norm");
    check(shc_mask_scores(P(), I32(), I64(), I32(), CODE(), P(), P(), P(), I32(), P(), P(), SZ(),
                          NULL),
          "mask_scores");
    check(shc_segment_maxpool(P(), P(), I64(), I32(), I32(), CODE(), PICK(kF), P(), NULL),
          "segment_maxpool");
    check(shc_transpose_neighbors(P(), I32(), I32(), P(), P(), (next_u64() & 1) ? &kt_host : NULL,
                                  P(), SZ(), NULL),
          "transpose_neighbors");
    check(shc_build_transposed_table(P(), P(), I64(), I32(), I32(), P(), I32(), P(), P(), NULL),
          "build_transposed_table");
    check(shc_sparse_linear_backward(P(), P(), P(), P(), I64(), I32(), I32(), CODE(), CODE(), P(),
                                     P(), P(), P(), SZ(), NULL),
          "sparse_linear_backward");
    check(shc_build_slot_pairs(P(), I64(), I32(), P(), P(), P(), SZ(), NULL), "build_slot_pairs");
    check(shc_sparse_neighbor_conv_backward(P(), P(), P(), P(), P(), P(), P(), I32(), P(), P(), P(),
                                            I64(), I32(), I32(), I32(), CODE(), CODE(), P(), P(),
                                            P(), P(), SZ(), NULL),
          "sparse_neighbor_conv_backward");
    check(shc_event_create((next_u64() & 1) ? &ev : NULL), "event_create");
    check(shc_event_record(NULL, NULL), "event_record");
    check(shc_stream_wait_event(NULL, NULL), "stream_wait_event");
    check(shc_event_synchronize(NULL), "event_synchronize");
    check(shc_event_destroy(NULL), "event_destroy");
  }
  printf("calls %ld ok %ld bad %d\n", g_calls, g_ok, g_bad);
  return g_bad;
}
