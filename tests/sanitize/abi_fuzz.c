/*
 * Host-side fuzz of the C ABI, built with AddressSanitizer and
 * UndefinedBehaviorSanitizer around the library's host code (abi.hip and
 * the stack executor, stack.hip).
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

/* A stack description: with probability 1/2 a coherent one (two bf16 conv
 * layers on a 4 x 655 batch, pipelined) with one to three fields then
 * replaced by edge values, else every field an edge value. */
static const int32_t kLayers[] = {-1, 0, 1, 2, 3, 16, 17};
static const int32_t kSets[] = {-1, 0, 1, 2, 3, 4};
static int64_t g_counts[3];

static void random_layer(shc_stack_layer* L) {
  L->kind = CODE();
  L->Cin = I32();
  L->Cout = I32();
  L->act = CODE();
  L->W = P();
  L->bias = P();
  L->plan_rows = I64();
  L->split_rows = I64();
}

static void random_set(shc_stack_index_set* x, int s) {
  x->coords = P();
  x->inv = P();
  x->row_ptr = P();
  x->n_active = P();
  x->host_count = (next_u64() & 1) ? &g_counts[s] : NULL;
  x->ws = P();
  x->ws_bytes = SZ();
  x->table = P();
  for (int l = 0; l < SHC_STACK_MAX_LAYERS; ++l) {
    x->plan[l] = P();
    x->plan_bytes[l] = SZ();
  }
}

static void stack_desc(shc_stack_desc* d) {
  memset(d, 0, sizeof *d);
  if (next_u64() & 1) {
    d->B = I32();
    d->V = I32();
    d->K = I32();
    d->dtype = CODE();
    d->C0 = I32();
    d->mask = P();
    d->x = P();
    d->nbr = P();
    d->table_in_compaction = CODE();
    d->n_layers = PICK(kLayers);
    for (int l = 0; l < SHC_STACK_MAX_LAYERS; ++l) random_layer(&d->layers[l]);
    for (int l = 0; l <= SHC_STACK_MAX_LAYERS; ++l) d->acts[l] = P();
    d->last_alt = P();
    d->dense_out = P();
    d->incremental = CODE();
    d->prev_coords = P();
    d->pooled = P();
    d->pool_empty = PICK(kF);
    d->n_sets = PICK(kSets);
    for (int s = 0; s < 3; ++s) random_set(&d->sets[s], s);
    d->side = (hipStream_t)P();
    d->tail = (hipStream_t)P();
    d->split_ws = P();
    d->split_ws_bytes = SZ();
    return;
  }
  /* coherent base; buffers at distinct aligned stand-in addresses */
  uintptr_t a = 0x100000;
#define NEXT() ((void*)(a += 0x1000))
  d->B = 4;
  d->V = 655;
  d->K = 9;
  d->dtype = SHC_BF16;
  d->C0 = 64;
  d->mask = NEXT();
  d->x = NEXT();
  d->nbr = NEXT();
  d->table_in_compaction = 1;
  d->n_layers = 2;
  for (int l = 0; l < 2; ++l) {
    shc_stack_layer* L = &d->layers[l];
    L->kind = SHC_LAYER_CONV;
    L->Cin = 64;
    L->Cout = 64;
    L->act = SHC_ACT_RELU;
    L->W = NEXT();
    L->bias = NULL;
    L->plan_rows = 1000;
  }
  for (int l = 0; l <= 2; ++l) d->acts[l] = NEXT();
  d->last_alt = NEXT();
  d->dense_out = NEXT();
  d->incremental = 1;
  d->prev_coords = NEXT();
  d->pooled = NEXT();
  d->n_sets = 3;
  for (int s = 0; s < 3; ++s) {
    shc_stack_index_set* x = &d->sets[s];
    x->coords = NEXT();
    x->inv = NEXT();
    x->row_ptr = NEXT();
    x->n_active = NEXT();
    x->host_count = &g_counts[s];
    x->ws = NEXT();
    x->ws_bytes = (size_t)1 << 20;
    x->table = NEXT();
    x->plan[0] = x->plan[1] = NEXT();
    x->plan_bytes[0] = x->plan_bytes[1] = (size_t)1 << 30;
  }
  d->side = (hipStream_t)NEXT();
  d->tail = (hipStream_t)NEXT();
  if (next_u64() & 1) {
    /* layer 1 by the split conv instead of its plan, with a workspace */
    d->layers[1].plan_rows = 0;
    d->layers[1].split_rows = 1000;
    for (int s = 0; s < 3; ++s) d->sets[s].plan[1] = NULL;
    d->split_ws = NEXT();
    d->split_ws_bytes = (size_t)1 << 30;
  }
#undef NEXT
  const int changes = 1 + (int)(next_u64() % 3);
  for (int c = 0; c < changes; ++c) {
    const int s = (int)(next_u64() % 3), l = (int)(next_u64() % 2);
    switch (next_u64() % 17) {
      case 0: d->B = I32(); break;
      case 1: d->V = I32(); break;
      case 2: d->K = I32(); break;
      case 3: d->dtype = CODE(); break;
      case 4: d->C0 = I32(); break;
      case 5: d->n_layers = PICK(kLayers); break;
      case 6: random_layer(&d->layers[l]); break;
      case 7: d->acts[next_u64() % 3] = P(); break;
      case 8: d->incremental = CODE(); d->prev_coords = P(); break;
      case 9: d->n_sets = PICK(kSets); break;
      case 10: random_set(&d->sets[s], s); break;
      case 11: d->sets[s].plan[l] = P(); d->sets[s].plan_bytes[l] = SZ(); break;
      case 12: d->side = (hipStream_t)P(); break;
      case 13: d->tail = d->side; break;
      case 14: d->table_in_compaction = CODE(); d->nbr = P(); break;
      case 15: d->split_ws = P(); d->split_ws_bytes = SZ(); break;
      default: d->sets[s].coords = d->sets[(s + 1) % 3].coords; break;
    }
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
    (void)shc_conv_split_workspace_bytes(I64(), I32(), I32(), I32(), CODE());
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
    check(shc_sparse_neighbor_conv_split(P(), P(), I64(), I32(), P(), P(), I32(), I32(), CODE(),
                                         CODE(), P(), P(), SZ(), NULL),
          "sparse_neighbor_conv_split");
    check(shc_sparse_neighbor_conv_planned(P(), P(), SZ(), I64(), I32(), P(), P(), I32(), I32(),
                                           CODE(), CODE(), P(), NULL),
          "sparse_neighbor_conv_planned");
    check(shc_scatter(P(), P(), P(), I64(), I32(), I32(), I32(), CODE(), CODE(), P(), NULL),
          "scatter");
    check(shc_scatter_update(P(), P(), P(), I64(), P(), I64(), I32(), I32(), I32(), CODE(), P(),
                             NULL),
          "scatter_update");
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
    shc_stack_desc desc;
    stack_desc(&desc);
    void* stk = NULL;
    check(shc_stack_create((next_u64() & 7) ? &desc : NULL, (next_u64() & 7) ? &stk : NULL),
          "stack_create");
    if (stk != NULL) {
      fprintf(stderr, "stack_create succeeded without a GPU\n");
      g_bad = 1;
      shc_stack_destroy(stk);
    }
    int32_t cur = (int32_t)(next_u64() % 5) - 1;
    int64_t prev = I64(), nl = 0;
    check(shc_stack_run(NULL, I64(), NULL, NULL, NULL, I32(), NULL, (next_u64() & 1) ? &cur : NULL,
                        &prev, &nl),
          "stack_run");
    check(shc_stack_destroy(NULL), "stack_destroy");
  }
  printf("calls %ld ok %ld bad %d\n", g_calls, g_ok, g_bad);
  return g_bad;
}
