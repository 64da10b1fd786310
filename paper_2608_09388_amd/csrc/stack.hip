// Stack executor: the whole sparse path (Sec. 3.2: compaction of a mask, the
// same active set through every layer, scatter and/or pool) over consecutive
// batches, issued from a native loop.  Every GPU step is one of the C ABI's
// own calls, enqueued in the order a caller of those calls would use; this
// file adds the schedule around them (index-set rotation, the streams and
// the events between them) and nothing else.
#include "../../include/shc.h"

#include <new>

#include "shc_internal.h"

namespace {

constexpr int kMaxSlots = 32;
constexpr int32_t kMaxChannels = 4096;

#define STK_TRY(expr)               \
  do {                              \
    int _rc = (expr);               \
    if (_rc != SHC_OK) return _rc;  \
  } while (0)

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int need_ptr(const void* p, const char* what, int idx = -1) {
  if (p == nullptr)
    return idx < 0 ? shc::set_error(SHC_ERR_INVALID_ARG, "%s is NULL", what)
                   : shc::set_error(SHC_ERR_INVALID_ARG, "%s[%d] is NULL", what, idx);
  if (!aligned16(p))
    return idx < 0 ? shc::set_error(SHC_ERR_MISALIGNED, "%s is not 16-byte aligned", what)
                   : shc::set_error(SHC_ERR_MISALIGNED, "%s[%d] is not 16-byte aligned", what,
                                    idx);
  return SHC_OK;
}

int opt_ptr(const void* p, const char* what, int idx = -1) {
  return p == nullptr ? SHC_OK : need_ptr(p, what, idx);
}

int hip_err(hipError_t e, const char* where) {
  if (e == hipSuccess) return SHC_OK;
  return shc::set_error(SHC_ERR_HIP, "%s: %s (%d)", where, hipGetErrorString(e), (int)e);
}

int check_channels(int32_t C, int l, const char* what) {
  if (C <= 0)
    return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: %s = %d must be positive", l, what, C);
  if (C % 16 != 0 || C > kMaxChannels)
    return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: %s = %d must be a multiple of 16 in "
                          "[16, %d]", l, what, C, kMaxChannels);
  return SHC_OK;
}

struct Stack {
  shc_stack_desc d;
  int device = -1;
  bool pipelined = false;
  bool fused_gather = false;  // layer 0 linear: shc_gather_sparse_linear
  bool has_conv = false;
  int32_t c_last = 0;
  // plan_owner[l] = l when layer l builds its plan each batch (the first
  // layer of the plan's buffer), another layer's index when it reads a plan
  // that layer builds, -1 without a plan
  int plan_owner[SHC_STACK_MAX_LAYERS];
  // stream-ordering events (device scope; see shc_event_create)
  hipEvent_t set_free[3] = {}, ready = nullptr, x_read = nullptr;
  hipEvent_t last_done[2] = {}, tail_done[2] = {}, tail_end = nullptr;
  bool busy = false;

  ~Stack() {
    for (hipEvent_t* e : {&set_free[0], &set_free[1], &set_free[2], &ready, &x_read,
                          &last_done[0], &last_done[1], &tail_done[0], &tail_done[1],
                          &tail_end})
      if (*e != nullptr) (void)hipEventDestroy(*e);
  }

  int64_t cap() const { return (int64_t)d.B * d.V; }

  // -- the calls of one batch on index set `s` -------------------------------
  int compact_start(int s, hipStream_t st) const {
    const shc_stack_index_set& x = d.sets[s];
    if (d.table_in_compaction)
      return shc_compact_mask_table_start(d.mask, d.B, d.V, x.coords, x.inv, x.row_ptr,
                                          x.n_active, x.host_count, cap(), d.nbr, d.K, x.table,
                                          x.ws, x.ws_bytes, st);
    return shc_compact_mask_start(d.mask, d.B, d.V, x.coords, x.inv, x.row_ptr, x.n_active,
                                  x.host_count, cap(), x.ws, x.ws_bytes, st);
  }

  int compact_wait(int s, hipStream_t st, int64_t* n) const {
    STK_TRY(shc_compact_mask_wait(d.sets[s].host_count, cap(), st));
    *n = *reinterpret_cast<volatile int64_t*>(d.sets[s].host_count);
    return SHC_OK;
  }

  // the neighbour-row table when the compaction did not write it
  int table(int s, int64_t n, hipStream_t st) const {
    if (!has_conv || d.table_in_compaction) return SHC_OK;
    const shc_stack_index_set& x = d.sets[s];
    return shc_build_neighbor_table(x.coords, x.inv, n, d.B, d.V, d.nbr, d.K, x.table, st);
  }

  bool planned(int l, int64_t n) const {
    return plan_owner[l] >= 0 && n > 0 && n <= d.layers[l].plan_rows;
  }

  bool split(int l, int64_t n) const { return n > 0 && n <= d.layers[l].split_rows; }

  bool packed(int l, int64_t n) const {
    return n > 0 && n >= d.layers[l].packed_min_rows && n <= d.layers[l].packed_rows;
  }

  int plans(int s, int64_t n, hipStream_t st) const {
    for (int l = 0; l < d.n_layers; ++l) {
      if (plan_owner[l] != l || !planned(l, n)) continue;
      const shc_stack_layer& L = d.layers[l];
      const shc_stack_index_set& x = d.sets[s];
      STK_TRY(shc_build_conv_plan(x.table, n, d.K, L.Cin, L.Cout, d.dtype, x.plan[l],
                                  x.plan_bytes[l], st));
    }
    return SHC_OK;
  }

  int gather(int s, int64_t n, hipStream_t st) const {
    if (fused_gather) return SHC_OK;
    return shc_gather_rows(d.x, d.sets[s].coords, n, d.B, d.V, d.C0, d.dtype, d.acts[0], st);
  }

  int layer(int s, int l, int64_t n, void* dst, hipStream_t st) const {
    const shc_stack_layer& L = d.layers[l];
    const shc_stack_index_set& x = d.sets[s];
    if (L.kind == SHC_LAYER_CONV) {
      if (packed(l, n))
        return shc_sparse_neighbor_conv_packed(d.acts[l], x.table, n, d.K, L.Wp, L.bias, L.Cin,
                                               L.Cout, d.dtype, L.act, dst, st);
      if (split(l, n))
        return shc_sparse_neighbor_conv_split(d.acts[l], x.table, n, d.K, L.W, L.bias, L.Cin,
                                              L.Cout, d.dtype, L.act, dst, d.split_ws,
                                              d.split_ws_bytes, st);
      if (planned(l, n))
        return shc_sparse_neighbor_conv_planned(d.acts[l], x.plan[l], x.plan_bytes[l], n, d.K,
                                                L.W, L.bias, L.Cin, L.Cout, d.dtype, L.act, dst,
                                                st);
      return shc_sparse_neighbor_conv_table(d.acts[l], x.table, n, d.K, L.W, L.bias, L.Cin,
                                            L.Cout, d.dtype, L.act, dst, st);
    }
    if (l == 0 && fused_gather)
      return shc_gather_sparse_linear(d.x, x.coords, n, d.B, d.V, L.W, L.bias, L.Cin, L.Cout,
                                      d.dtype, L.act, dst, st);
    return shc_sparse_linear(d.acts[l], n, L.W, L.bias, L.Cin, L.Cout, d.dtype, L.act, dst, st);
  }

  // scatter (zero-fill, or the update of the previous batch's output) and pool
  int finish(int s, int64_t n, const void* src, hipStream_t st, int64_t* prev_rows) const {
    const shc_stack_index_set& x = d.sets[s];
    if (d.dense_out != nullptr) {
      if (d.incremental) {
        STK_TRY(shc_scatter_update(src, x.inv, x.coords, n, d.prev_coords, *prev_rows, d.B,
                                   d.V, c_last, d.dtype, d.dense_out, st));
        if (n > 0)
          STK_TRY(hip_err(hipMemcpyAsync(d.prev_coords, x.coords, (size_t)n * 2 * sizeof(int32_t),
                                         hipMemcpyDeviceToDevice, st),
                          "stack: copy of the scattered coordinates"));
        *prev_rows = n;
      } else {
        STK_TRY(shc_scatter(src, x.inv, x.coords, n, d.B, d.V, c_last, d.dtype, 1, d.dense_out,
                            st));
      }
    }
    if (d.pooled != nullptr)
      STK_TRY(shc_segment_maxpool(src, x.row_ptr, n, d.B, c_last, d.dtype, d.pool_empty,
                                  d.pooled, st));
    return SHC_OK;
  }

  // -- schedules -------------------------------------------------------------
  struct RunArgs {
    int64_t steps;
    hipStream_t main;
    shc_stack_feed_fn feed;
    void* user;
    int32_t time_layer;
    void* const* time_events;
  };

  int feed_batch(const RunArgs& a, int64_t k, hipStream_t st) const {
    if (a.feed == nullptr) return SHC_OK;
    const int r = a.feed(a.user, k, st);
    if (r != 0)
      return shc::set_error(SHC_ERR_INVALID_ARG, "stack: feed of batch %lld returned %d",
                            (long long)k, r);
    return SHC_OK;
  }

  int record_time(const RunArgs& a, int64_t k, int which, int l) const {
    if (a.time_events == nullptr || l != a.time_layer) return SHC_OK;
    void* e = a.time_events[2 * k + which];
    if (e == nullptr) return SHC_OK;
    return hip_err(hipEventRecord(static_cast<hipEvent_t>(e), a.main), "stack: timing event");
  }

  // every layer of batch k on set s (the last one into `last`)
  int layers(const RunArgs& a, int64_t k, int s, int64_t n, void* last, hipStream_t st,
             hipEvent_t before_last, hipEvent_t after_first) const {
    for (int l = 0; l < d.n_layers; ++l) {
      void* dst = d.acts[l + 1];
      if (l == d.n_layers - 1) {
        if (before_last != nullptr)
          STK_TRY(hip_err(hipStreamWaitEvent(st, before_last, 0), "stack: wait"));
        dst = last;
      }
      STK_TRY(record_time(a, k, 0, l));
      STK_TRY(layer(s, l, n, dst, st));
      STK_TRY(record_time(a, k, 1, l));
      if (l == 0 && fused_gather && after_first != nullptr)
        STK_TRY(hip_err(hipEventRecord(after_first, st), "stack: record"));
    }
    return SHC_OK;
  }

  // one stream: compaction of batch k + 1 before the scatter and pool of batch k
  int run_serial(const RunArgs& a, int* cur, int64_t* prev_rows, int64_t* n_last) const {
    hipStream_t st = a.main;
    int s = *cur;
    int64_t n = 0;
    STK_TRY(feed_batch(a, 0, st));
    STK_TRY(compact_start(s, st));
    STK_TRY(compact_wait(s, st, &n));
    for (int64_t k = 0; k < a.steps; ++k) {
      STK_TRY(table(s, n, st));
      STK_TRY(plans(s, n, st));
      STK_TRY(gather(s, n, st));
      STK_TRY(layers(a, k, s, n, d.acts[d.n_layers], st, nullptr, nullptr));
      int nxt = -1;
      if (k + 1 < a.steps) {
        nxt = (s + 1) % d.n_sets;
        STK_TRY(feed_batch(a, k + 1, st));
        STK_TRY(compact_start(nxt, st));
      }
      STK_TRY(finish(s, n, d.acts[d.n_layers], st, prev_rows));
      if (nxt >= 0) {
        STK_TRY(compact_wait(nxt, st, &n));
        s = nxt;
      }
    }
    *cur = s;
    *n_last = n;
    return SHC_OK;
  }

  // three streams: batch k's layers on the run's stream, batch k + 1's
  // compaction (table, plans) on the side stream, batch k's scatter and pool
  // on the tail stream; the last layer's output alternates between two
  // buffers and the index sets rotate over three
  int run_pipelined(const RunArgs& a, int* cur, int64_t* prev_rows, int64_t* n_last) const {
    hipStream_t main = a.main, side = d.side, tail = d.tail;
    bool set_used[3] = {false, false, false};
    bool buf_used[2] = {false, false};
    void* const last_buf[2] = {d.acts[d.n_layers], d.last_alt};
    const bool feeding = a.feed != nullptr;
    int s = *cur;
    int64_t n = 0;
    STK_TRY(feed_batch(a, 0, main));
    STK_TRY(compact_start(s, main));
    STK_TRY(compact_wait(s, main, &n));
    bool front_done = false;  // table and plans of set s already built (side stream)
    for (int64_t k = 0; k < a.steps; ++k) {
      const int i = (int)((a.steps - 1 - k) % 2);  // the last batch writes acts[n_layers]
      if (!front_done) {
        STK_TRY(table(s, n, main));
        STK_TRY(plans(s, n, main));
      }
      STK_TRY(gather(s, n, main));
      if (!fused_gather && feeding)
        STK_TRY(hip_err(hipEventRecord(x_read, main), "stack: record"));
      STK_TRY(layers(a, k, s, n, last_buf[i], main, buf_used[i] ? tail_done[i] : nullptr,
                     feeding ? x_read : nullptr));
      STK_TRY(hip_err(hipEventRecord(last_done[i], main), "stack: record"));
      buf_used[i] = true;
      // compaction of batch k + 1 (side stream)
      int nxt = -1;
      if (k + 1 < a.steps) {
        nxt = (s + 1) % 3;
        if (feeding) {
          // batch k + 1's inputs are written once batch k's gather has read x
          // (batch k's compaction read the mask earlier on this stream)
          STK_TRY(hip_err(hipStreamWaitEvent(side, x_read, 0), "stack: wait"));
          STK_TRY(feed_batch(a, k + 1, side));
        }
        // the set was last read by the scatter and pool of batch k - 2
        if (set_used[nxt])
          STK_TRY(hip_err(hipEventSynchronize(set_free[nxt]), "stack: set reuse wait"));
        STK_TRY(compact_start(nxt, side));
      }
      // scatter and pool of batch k (tail stream)
      STK_TRY(hip_err(hipStreamWaitEvent(tail, last_done[i], 0), "stack: wait"));
      STK_TRY(finish(s, n, last_buf[i], tail, prev_rows));
      STK_TRY(hip_err(hipEventRecord(tail_done[i], tail), "stack: record"));
      STK_TRY(hip_err(hipEventRecord(set_free[s], tail), "stack: record"));
      set_used[s] = true;
      if (nxt >= 0) {
        int64_t n_next = 0;
        STK_TRY(compact_wait(nxt, side, &n_next));
        STK_TRY(table(nxt, n_next, side));
        STK_TRY(plans(nxt, n_next, side));
        front_done = true;
        STK_TRY(hip_err(hipEventRecord(ready, side), "stack: record"));
        STK_TRY(hip_err(hipStreamWaitEvent(main, ready, 0), "stack: wait"));
        s = nxt;
        n = n_next;
      }
    }
    STK_TRY(hip_err(hipEventRecord(tail_end, tail), "stack: record"));
    STK_TRY(hip_err(hipStreamWaitEvent(main, tail_end, 0), "stack: wait"));
    *cur = s;
    *n_last = n;
    return SHC_OK;
  }
};

// Every check the run's calls would make, done once at creation.
int check_desc(const shc_stack_desc& d, Stack* k) {
  if (d.B <= 0 || d.V <= 0)
    return shc::set_error(SHC_ERR_INVALID_ARG, "B = %d and V = %d must be positive", d.B, d.V);
  if ((int64_t)d.B * d.V > INT32_MAX)
    return shc::set_error(SHC_ERR_UNSUPPORTED, "B * V = %lld exceeds 2^31 - 1",
                          (long long)d.B * d.V);
  if (d.dtype != SHC_F32 && d.dtype != SHC_BF16)
    return shc::set_error(SHC_ERR_UNSUPPORTED, "unknown dtype code %d", d.dtype);
  if (d.n_layers < 1 || d.n_layers > SHC_STACK_MAX_LAYERS)
    return shc::set_error(SHC_ERR_INVALID_ARG, "n_layers = %d outside [1, %d]", d.n_layers,
                          SHC_STACK_MAX_LAYERS);
  STK_TRY(need_ptr(d.mask, "mask"));
  STK_TRY(need_ptr(d.x, "x"));
  STK_TRY(check_channels(d.C0, 0, "C0"));
  k->has_conv = false;
  int32_t c_prev = d.C0;
  size_t split_need = 0;  // the largest split workspace of any layer
  for (int l = 0; l < d.n_layers; ++l) {
    const shc_stack_layer& L = d.layers[l];
    if (L.kind != SHC_LAYER_LINEAR && L.kind != SHC_LAYER_CONV)
      return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: unknown kind %d", l, L.kind);
    STK_TRY(check_channels(L.Cin, l, "Cin"));
    STK_TRY(check_channels(L.Cout, l, "Cout"));
    if (L.Cin != c_prev)
      return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: Cin = %d but its input has %d "
                            "channels", l, L.Cin, c_prev);
    c_prev = L.Cout;
    if (L.act != SHC_ACT_NONE && L.act != SHC_ACT_RELU)
      return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: unknown act code %d", l, L.act);
    STK_TRY(need_ptr(L.W, "layers.W", l));
    STK_TRY(opt_ptr(L.bias, "layers.bias", l));
    if (L.plan_rows < 0)
      return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: plan_rows = %lld is negative", l,
                            (long long)L.plan_rows);
    if (L.split_rows < 0)
      return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: split_rows = %lld is negative", l,
                            (long long)L.split_rows);
    if (L.packed_min_rows < 0)
      return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: packed_min_rows = %lld is negative",
                            l, (long long)L.packed_min_rows);
    if (L.packed_rows < 0)
      return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: packed_rows = %lld is negative", l,
                            (long long)L.packed_rows);
    if (L.packed_rows > 0) {
      if (L.kind != SHC_LAYER_CONV)
        return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: a linear layer takes no packed "
                              "conv", l);
      if (L.plan_rows > 0 || L.split_rows > 0)
        return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: packed_rows with plan_rows or "
                              "split_rows", l);
      if (shc_conv_packed_weights_bytes(d.K, L.Cin, L.Cout, d.dtype) == 0)
        return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: no packed conv for this shape", l);
      if ((int64_t)d.K * L.packed_rows * 4 > 0x7FFFFFFFLL)
        return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: packed_rows = %lld too large", l,
                              (long long)L.packed_rows);
      STK_TRY(need_ptr(L.Wp, "layers.Wp", l));
    }
    if (L.split_rows > 0) {
      if (L.kind != SHC_LAYER_CONV)
        return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: a linear layer takes no split "
                              "conv", l);
      if (L.plan_rows > 0)
        return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: plan_rows and split_rows both "
                              "set", l);
      const size_t need = shc_conv_split_workspace_bytes(L.split_rows, d.K, L.Cin, L.Cout,
                                                         d.dtype);
      if (need == 0)
        return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: no split conv for %lld rows of "
                              "this shape", l, (long long)L.split_rows);
      split_need = need > split_need ? need : split_need;
    }
    if (L.kind == SHC_LAYER_CONV) {
      k->has_conv = true;
      if (L.plan_rows > 0) {
        const int64_t lim = shc_conv_plan_max_rows(d.K, L.Cin, L.Cout, d.dtype);
        if (L.plan_rows > lim)
          return shc::set_error(SHC_ERR_UNSUPPORTED, "layer %d: plan_rows = %lld above the "
                                "%lld rows a plan of this shape takes", l,
                                (long long)L.plan_rows, (long long)lim);
      }
    } else if (L.plan_rows != 0) {
      return shc::set_error(SHC_ERR_INVALID_ARG, "layer %d: a linear layer takes no plan", l);
    }
    STK_TRY(need_ptr(d.acts[l + 1], "acts", l + 1));
  }
  k->c_last = c_prev;
  if (split_need > 0) {
    STK_TRY(need_ptr(d.split_ws, "split_ws"));
    if (d.split_ws_bytes < split_need)
      return shc::set_error(SHC_ERR_CAPACITY, "split_ws_bytes = %zu is below the %zu bytes the "
                            "split layers need", d.split_ws_bytes, split_need);
  } else if (d.split_ws != nullptr) {
    return shc::set_error(SHC_ERR_INVALID_ARG, "split_ws given but no layer has split_rows > 0");
  }
  k->fused_gather = d.layers[0].kind == SHC_LAYER_LINEAR;
  if (!k->fused_gather) STK_TRY(need_ptr(d.acts[0], "acts", 0));
  if (k->has_conv) {
    if (d.K <= 0) return shc::set_error(SHC_ERR_INVALID_ARG, "K = %d must be positive", d.K);
    if (d.K > kMaxSlots)
      return shc::set_error(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", d.K, kMaxSlots);
    STK_TRY(need_ptr(d.nbr, "nbr"));
  }
  if (d.table_in_compaction != 0 && d.table_in_compaction != 1)
    return shc::set_error(SHC_ERR_INVALID_ARG, "table_in_compaction = %d must be 0 or 1",
                          d.table_in_compaction);
  if (d.table_in_compaction && !k->has_conv)
    return shc::set_error(SHC_ERR_INVALID_ARG, "table_in_compaction without a conv layer");
  if (d.table_in_compaction && !shc::compact_table_supported(d.V, d.K))
    return shc::set_error(SHC_ERR_UNSUPPORTED, "V = %d, K = %d: the compaction cannot write "
                          "the table", d.V, d.K);
  if (d.incremental != 0 && d.incremental != 1)
    return shc::set_error(SHC_ERR_INVALID_ARG, "incremental = %d must be 0 or 1", d.incremental);
  STK_TRY(opt_ptr(d.dense_out, "dense_out"));
  STK_TRY(opt_ptr(d.pooled, "pooled"));
  if (d.incremental) {
    if (d.dense_out == nullptr)
      return shc::set_error(SHC_ERR_INVALID_ARG, "incremental scatter without dense_out");
    STK_TRY(need_ptr(d.prev_coords, "prev_coords"));
  }
  if ((d.side == nullptr) != (d.tail == nullptr))
    return shc::set_error(SHC_ERR_INVALID_ARG, "side and tail streams must both be set or "
                          "both be NULL");
  k->pipelined = d.side != nullptr;
  if (k->pipelined) {
    if (d.side == d.tail)
      return shc::set_error(SHC_ERR_INVALID_ARG, "side and tail must be different streams");
    if (d.n_sets != 3)
      return shc::set_error(SHC_ERR_INVALID_ARG, "a pipelined stack takes 3 index sets, "
                            "not %d", d.n_sets);
    STK_TRY(need_ptr(d.last_alt, "last_alt"));
  } else if (d.n_sets != 2 && d.n_sets != 3) {
    return shc::set_error(SHC_ERR_INVALID_ARG, "n_sets = %d must be 2 or 3", d.n_sets);
  }
  const size_t ws_need = shc_compact_mask_workspace(d.B, d.V);
  for (int s = 0; s < d.n_sets; ++s) {
    const shc_stack_index_set& x = d.sets[s];
    STK_TRY(need_ptr(x.coords, "sets.coords", s));
    STK_TRY(need_ptr(x.inv, "sets.inv", s));
    STK_TRY(need_ptr(x.row_ptr, "sets.row_ptr", s));
    STK_TRY(need_ptr(x.n_active, "sets.n_active", s));
    STK_TRY(need_ptr(x.ws, "sets.ws", s));
    if (x.host_count == nullptr)
      return shc::set_error(SHC_ERR_INVALID_ARG, "sets.host_count[%d] is NULL", s);
    if (x.ws_bytes < ws_need)
      return shc::set_error(SHC_ERR_CAPACITY, "sets.ws[%d]: %zu bytes, below the %zu needed",
                            s, x.ws_bytes, ws_need);
    if (k->has_conv) STK_TRY(need_ptr(x.table, "sets.table", s));
    if (d.incremental && x.coords == d.prev_coords)
      return shc::set_error(SHC_ERR_INVALID_ARG, "prev_coords is index set %d's coords", s);
    for (int t = 0; t < s; ++t)
      if (d.sets[t].coords == x.coords || d.sets[t].inv == x.inv ||
          d.sets[t].host_count == x.host_count)
        return shc::set_error(SHC_ERR_INVALID_ARG, "index sets %d and %d share a buffer", t, s);
    for (int l = 0; l < d.n_layers; ++l) {
      const shc_stack_layer& L = d.layers[l];
      const bool wants = L.kind == SHC_LAYER_CONV && L.plan_rows > 0;
      if (!wants) {
        if (x.plan[l] != nullptr)
          return shc::set_error(SHC_ERR_INVALID_ARG, "sets.plan[%d][%d] given to a layer with "
                                "plan_rows = 0", s, l);
        continue;
      }
      STK_TRY(need_ptr(x.plan[l], "sets.plan", l));
      const size_t nb = shc_conv_plan_bytes(L.plan_rows, d.K, L.Cin, L.Cout, d.dtype);
      if (x.plan_bytes[l] < nb)
        return shc::set_error(SHC_ERR_CAPACITY, "sets.plan_bytes[%d][%d] = %zu, below the %zu "
                              "a plan of %lld rows takes", s, l, x.plan_bytes[l], nb,
                              (long long)L.plan_rows);
      for (int m = 0; m < l; ++m)
        if (x.plan[m] == x.plan[l] &&
            (d.layers[m].Cin != L.Cin || d.layers[m].Cout != L.Cout ||
             d.layers[m].plan_rows != L.plan_rows))
          return shc::set_error(SHC_ERR_INVALID_ARG, "layers %d and %d share a plan buffer but "
                                "not its shape and row limit", m, l);
    }
  }
  // which layer builds each plan: the first layer of a buffer (same in every
  // set: sharing is checked on set 0's pointers and must match elsewhere)
  for (int l = 0; l < d.n_layers; ++l) {
    k->plan_owner[l] = -1;
    if (d.sets[0].plan[l] == nullptr) continue;
    k->plan_owner[l] = l;
    for (int m = 0; m < l; ++m)
      if (d.sets[0].plan[m] == d.sets[0].plan[l]) {
        k->plan_owner[l] = k->plan_owner[m];
        break;
      }
    for (int s = 1; s < d.n_sets; ++s)
      if (d.sets[s].plan[k->plan_owner[l]] != d.sets[s].plan[l])
        return shc::set_error(SHC_ERR_INVALID_ARG, "index set %d shares plan buffers "
                              "differently from set 0 (layer %d)", s, l);
  }
  return SHC_OK;
}

}  // namespace

extern "C" {

int shc_stack_create(const shc_stack_desc* desc, void** stack) {
  shc::clear_error();
  if (stack == nullptr) return shc::set_error(SHC_ERR_INVALID_ARG, "stack is NULL");
  *stack = nullptr;
  if (desc == nullptr) return shc::set_error(SHC_ERR_INVALID_ARG, "desc is NULL");
  Stack* k = new (std::nothrow) Stack();
  if (k == nullptr) return shc::set_error(SHC_ERR_INVALID_ARG, "out of host memory");
  k->d = *desc;
  int rc = check_desc(k->d, k);
  // the host counts must be page-locked and mapped (the compaction refuses
  // them otherwise, which would stop a run after its first batch)
  for (int s = 0; rc == SHC_OK && s < k->d.n_sets; ++s) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, k->d.sets[s].host_count) != hipSuccess ||
        attr.type != hipMemoryTypeHost || attr.devicePointer == nullptr) {
      (void)hipGetLastError();
      rc = shc::set_error(SHC_ERR_INVALID_ARG, "sets.host_count[%d] is not page-locked host "
                          "memory mapped into the device", s);
    }
  }
  if (rc == SHC_OK) rc = hip_err(hipGetDevice(&k->device), "stack: current device");
  const unsigned flags = hipEventDisableTiming | hipEventDisableSystemFence;
  for (hipEvent_t* e : {&k->set_free[0], &k->set_free[1], &k->set_free[2], &k->ready,
                        &k->x_read, &k->last_done[0], &k->last_done[1], &k->tail_done[0],
                        &k->tail_done[1], &k->tail_end})
    if (rc == SHC_OK) rc = hip_err(hipEventCreateWithFlags(e, flags), "stack: event create");
  if (rc != SHC_OK) {
    delete k;
    return rc;
  }
  *stack = k;
  return SHC_OK;
}

int shc_stack_run(void* stack, int64_t steps, hipStream_t stream, shc_stack_feed_fn feed,
                  void* user, int32_t time_layer, void* const* time_events, int32_t* cur_set,
                  int64_t* prev_rows, int64_t* n_last) {
  shc::clear_error();
  if (stack == nullptr) return shc::set_error(SHC_ERR_INVALID_ARG, "stack is NULL");
  if (cur_set == nullptr || prev_rows == nullptr || n_last == nullptr)
    return shc::set_error(SHC_ERR_INVALID_ARG, "cur_set, prev_rows and n_last must be given");
  Stack* k = static_cast<Stack*>(stack);
  if (steps < 0)
    return shc::set_error(SHC_ERR_INVALID_ARG, "steps = %lld is negative", (long long)steps);
  if (*cur_set < 0 || *cur_set >= k->d.n_sets)
    return shc::set_error(SHC_ERR_INVALID_ARG, "cur_set = %d outside [0, %d)", *cur_set,
                          k->d.n_sets);
  if (*prev_rows < 0 || *prev_rows > k->cap())
    return shc::set_error(SHC_ERR_INVALID_ARG, "prev_rows = %lld outside [0, B*V]",
                          (long long)*prev_rows);
  if (time_events != nullptr && (time_layer < 0 || time_layer >= k->d.n_layers))
    return shc::set_error(SHC_ERR_INVALID_ARG, "time_layer = %d outside [0, %d)", time_layer,
                          k->d.n_layers);
  if (k->pipelined && (stream == k->d.side || stream == k->d.tail))
    return shc::set_error(SHC_ERR_INVALID_ARG, "the run's stream is the side or tail stream");
  int dev = -1;
  STK_TRY(hip_err(hipGetDevice(&dev), "stack: current device"));
  if (dev != k->device)
    return shc::set_error(SHC_ERR_INVALID_ARG, "current device %d, stack created on %d", dev,
                          k->device);
  if (k->busy) return shc::set_error(SHC_ERR_INVALID_ARG, "the stack is already running");
  if (steps == 0) {
    *n_last = 0;
    return SHC_OK;
  }
  k->busy = true;
  const Stack::RunArgs a{steps, stream, feed, user, time_layer, time_events};
  int cur = *cur_set;
  int64_t prev = *prev_rows;
  const int rc = k->pipelined ? k->run_pipelined(a, &cur, &prev, n_last)
                              : k->run_serial(a, &cur, &prev, n_last);
  k->busy = false;
  *cur_set = cur;
  *prev_rows = prev;
  return rc;
}

int shc_stack_destroy(void* stack) {
  shc::clear_error();
  delete static_cast<Stack*>(stack);
  return SHC_OK;
}

}  // extern "C"
