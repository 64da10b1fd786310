// Weight-stationary gathered-row contraction: the sparse neighbourhood
// convolution (Eqs. 4-5) and the sparse linear layer (Eq. 6) for the shapes
// where a column slice of the weights fits in LDS.
//
// The computed quantity is the same as in gemm.hip:
//
//   out[i][n] = act( bias[n] + sum_{j<K} sum_{c<Cin} S[r_ij][c] * W[j][c][n] ),
//
// with r_ij = inv[b_i*V + nbr[v_i*K + j]] (conv) or i (linear, K = 1), and a
// slot with r_ij = -1 adding nothing.
//
// Organisation (one workgroup = 8 wavefronts = 512 threads, one per CU):
//   * the grid is (row groups) x (column slices of width WS).  A workgroup
//     copies W[:, :, slice] (all K*Cin reduction rows) into LDS once and keeps
//     it there, so the weights cross the memory system once per workgroup;
//   * it builds the index lists of its whole row range with three rounds of
//     loads (coordinates, neighbour vertices, inverse-map rows), each round
//     fully in flight, while the weight slice streams in alongside;
//   * the rows are bucketed (LDS histogram and cursors) by their first
//     sparse slot -- a slot present in fewer than half of the rows.  16-row
//     blocks then hold rows with only dense slots, or rows sharing a sparse
//     slot, and each block carries the set of slots any of its rows has;
//   * every wavefront walks its list of jobs (block, live slot), built once,
//     over blocks b = wave, wave + 8, ...  A job loads the A fragments of its
//     slot (16 bytes per lane of the gathered neighbour rows, one per 64-byte
//     k-step) with raw buffer loads, an absent row reading zeros; jobs are
//     issued D ahead through a ring of register sets.  All B fragments of a
//     job are read from the resident slice (ds_read_b64_tr_b16 for bf16)
//     before its MFMAs (one per 16 output columns).  No barrier in this loop;
//   * accumulators start at the bias; when a block's last job is done its 16
//     rows x WS columns get the activation and the rounding, and go back
//     through a per-wave LDS scratch as 16-byte vectors to the rows' original
//     positions.
// Every output row is accumulated over the same (slot, k-step) sequence
// whatever block it lands in (absent slots contribute exact zeros), so the
// result does not depend on the order the sort produced.
#include <algorithm>
#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

// 8 wavefronts (two per SIMD) for both; 12 for the conv fit its registers
// but measured slower (more loads in flight contend in the memory path)
constexpr int kThreadsConv = 512;
constexpr int kThreadsLin = 512;
constexpr int kMaxSlots = 32;
constexpr int kBuckets = kMaxSlots + 2;
constexpr int kMaxRows = 1536;                // rows per workgroup
constexpr int kLdsLimit = 160 * 1024;
constexpr int kWBatch = 8;                    // weight vectors in flight per thread
// jobs of one wavefront: at most kMaxRows / 16 / waves blocks of at most 10 live slots
constexpr int kMaxJobs = 128;
static_assert((kMaxRows / 16 + 7) / 8 * 10 <= kMaxJobs, "job list too short");
static_assert(kMaxRows % kThreadsConv == 0 && kMaxRows % kThreadsLin == 0, "rows per thread");

typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
// third word of a raw buffer resource on gfx9-family parts (32-bit data, no swizzle)
constexpr int kBufferWord3 = 0x00020000;
// a buffer offset past any buffer the kernel is given (buffers are < 2 GiB)
constexpr uint32_t kOutOfRange = 0x80000000u;
#define SHC_LDS __attribute__((address_space(3)))

template <bool BF16>
struct WElem;
template <>
struct WElem<true> {
  static constexpr int bytes = 2;
  static constexpr int per_vec = 8;
  static constexpr int kstep = 32;  // entries per MFMA k-step (64 bytes)
};
template <>
struct WElem<false> {
  static constexpr int bytes = 4;
  static constexpr int per_vec = 4;
  static constexpr int kstep = 16;
};

// epilogue staging row (padded)
__host__ __device__ inline int ws_wrow(int ws, int e) { return ws * e + 16; }
// weight-slice row: unpadded for bf16 (the 32-byte column chunks are
// XOR-swizzled instead, see swz_chunk), padded for fp32
__host__ __device__ inline int ws_wrow_w(int ws, int e) { return e == 2 ? ws * e : ws * e + 16; }
// srcs[rows*K], perm[rows], blkmask[rows/16], scnt[waves][kMaxSlots],
// bcnt[kBuckets][kRPT][waves] (counts, then exclusive starts, in scan order),
// jobl[waves][kMaxJobs] (each wavefront's job list)
__host__ __device__ inline int ws_idx_bytes(int rows, int K, int waves, int rpt) {
  return (4 * (rows * K + rows + rows / 16 + waves * kMaxSlots + rpt * waves * kBuckets +
               waves * kMaxJobs) +
          15) & ~15;
}
// epilogue staging for every wave, then one k-step of zero weight rows
__host__ __device__ inline int ws_scratch(int ws, int e, int waves) {
  return waves * 16 * ws_wrow(ws, e) + (e == 2 ? 32 : 16) * ws_wrow_w(ws, e);
}

// KM: slots held per row in registers during the index build (>= K).
// KSM: k-steps per slot held per job (>= Cin / kstep); D jobs in flight.
// 16 bytes per lane from global memory straight into LDS: lane i's vector
// lands at dst + 16 i (dst is the wavefront's LDS base)
__device__ __forceinline__ void lds_direct_load16(const void* src, SHC_LDS void* dst) {
  __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
}

// DW: the weight slice goes straight into LDS with 16-byte direct loads, all
// issued first (bf16, full column slices, a multiple of 64 vectors; conv from
// a table, or linear).
// MODE (conv from a table, bf16, direct weight loads only):
//   kFull    -- everything in one launch;
//   kPlanOut -- the index lists, sort and job lists of one row group, without
//               the weights, copied from LDS to plan + blockIdx.x * plan_stride
//               (the "plan" of the active set: the same for every column slice
//               and every layer of the same shape on it);
//   kPlanned -- the index lists come from such a plan (16-byte direct loads
//               into LDS beside the weight slice) instead of the table.
constexpr int kFull = 0, kPlanOut = 1, kPlanned = 2;
template <bool BF16, int WS, bool CONV, bool TBL, int KM, int KSM, bool DW = false,
          int MODE = kFull>
__global__ __launch_bounds__(CONV ? kThreadsConv : kThreadsLin, 1) void ws_kernel(GemmArgs a,
                                                                                   int R) {
  static_assert(MODE == kFull || (BF16 && CONV && TBL && DW), "plans: bf16 table conv only");
  constexpr int kThreads = CONV ? kThreadsConv : kThreadsLin;
  constexpr int kWaves = kThreads / 64;
  constexpr int kRPT = kMaxRows / kThreads;  // rows per thread in the index build
  using E = WElem<BF16>;
  constexpr int NCB = WS / 16;             // 16-column blocks in the slice
  constexpr int WROW = WS * E::bytes + 16;        // epilogue staging row
  constexpr int WROWW = BF16 ? WS * 2 : WROW;      // weight-slice row
  constexpr int VPR = WS * E::bytes / 16;  // 16-byte vectors per slice row
  // jobs in flight (fewer when the linear layer keeps its B fragments in registers)
  constexpr int D = (BF16 && !CONV && KSM * NCB <= 32) ? 12 / KSM : 16 / KSM;

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int K = CONV ? a.K : 1;
  const int Cin = a.Cin;
  const int Cout = a.Cout;
  const int Ktot = K * Cin;
  const int KS = Cin / E::kstep;  // k-steps per slot (Cin * e is a multiple of 64)

  unsigned char* wl = smem;  // [Ktot][WROWW] (none in a plan build)
  const int wbytes = MODE == kPlanOut ? 0 : (Ktot * WROWW + 15) & ~15;
  int32_t* srcs = reinterpret_cast<int32_t*>(smem + wbytes);    // [R][K], sorted order
  int32_t* perm = srcs + R * K;                                 // [R] position -> row
  uint32_t* blkmask = reinterpret_cast<uint32_t*>(perm + R);    // [R/16]
  int32_t* scnt = reinterpret_cast<int32_t*>(blkmask + R / 16); // [waves][kMaxSlots]
  int32_t* bcnt = scnt + kWaves * kMaxSlots;                    // [kBuckets][kRPT][waves]
  int32_t* jobl = bcnt + kBuckets * kRPT * kWaves;              // [waves][kMaxJobs]
  unsigned char* scratch = smem + wbytes + ws_idx_bytes(R, K, kWaves, kRPT);  // [waves][16][WROW]
  unsigned char* zrows = scratch + kWaves * 16 * WROW;           // [kstep][WROWW] zeros

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 4;
  const int l16 = lane & 15;

  const int64_t row0 = (int64_t)blockIdx.x * R;
  const int nrows = (int)min((int64_t)R, a.n_rows - row0);
  const int nblk = (nrows + 15) / 16;
  const int n0 = blockIdx.y * WS;
  const unsigned char* W = static_cast<const unsigned char*>(a.W);
  // bias of this lane's columns, loaded now so the prologue hides the latency
  // (the selection below waits until after it)
  // (a plan build has neither weights nor bias)
  float bias_raw[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int col = n0 + cb * 16 + l16;
    const float* bp = a.bias != nullptr ? a.bias : reinterpret_cast<const float*>(a.W);
    bias_raw[cb] = MODE == kPlanOut ? 0.f : bp[(a.bias != nullptr && col < Cout) ? col : 0];
  }

  // Byte offset of 16-byte vector q in weight-slice row k.  For bf16 the
  // 32-byte column chunk (16 output columns) is XOR-ed with bit 1 ^ bit 3 of
  // the row: the transposing reads of a wavefront then touch rows r and r + 8
  // (and r, r + 2) in different chunks, so no two lanes of a cycle share an
  // LDS bank.  For a reduction row 8g + i (+4) of a 32-row k-step the swizzle
  // bit is ((i >> 1) ^ g) & 1, a per-lane constant (swz_lane).
  auto w_col = [&](int k, int q) -> int {
    if (!BF16 || NCB < 2) return q * 16;
    const int h = ((k >> 1) ^ (k >> 3)) & 1;
    return ((((q >> 1) ^ h)) << 5) + ((q & 1) << 4);
  };
  const int swz_lane = (BF16 && NCB >= 2) ? ((((l16 >> 2) >> 1) ^ g) & 1) : 0;

  // ---- weight slice W[k][n0 .. n0 + WS) -> LDS, kWBatch vectors per thread at a time
  const int wvecs = Ktot * VPR;
  auto load_w = [&](int base, i32x4* wv) {
#pragma unroll
    for (int u = 0; u < kWBatch; ++u) {
      const int v = base + u * kThreads + tid;
      const int k = v / VPR;
      const int q = v - k * VPR;
      const int n = n0 + q * E::per_vec;
      const bool ok = v < wvecs && n < Cout;
      wv[u] = *reinterpret_cast<const i32x4*>(
          W + (ok ? ((int64_t)k * Cout + n) * E::bytes : 0));
      if (!ok) wv[u] = i32x4{0, 0, 0, 0};
    }
  };
  auto store_w = [&](int base, const i32x4* wv) {
#pragma unroll
    for (int u = 0; u < kWBatch; ++u) {
      const int v = base + u * kThreads + tid;
      const int k = v / VPR;
      const int q = v - k * VPR;
      if (v < wvecs) *reinterpret_cast<i32x4*>(wl + k * WROWW + w_col(k, q)) = wv[u];
    }
  };
  i32x4 wv[kWBatch];
  if constexpr (MODE == kPlanOut) {
    // no weights in a plan
  } else if constexpr (DW) {
    // LDS vector v = 64 c + lane of the slice is row k = v / VPR, position
    // p = v % VPR; it holds source vector q with w_col(k, q) = 16 p (the
    // chunk swizzle is its own inverse).  A wavefront's direct load writes
    // 64 consecutive vectors; the waits come before the prologue's last barrier.
    for (int c = wave; c < wvecs / 64; c += kWaves) {
      const int v = c * 64 + lane;
      const int k = v / VPR;
      const int p = v - k * VPR;
      const int h = ((k >> 1) ^ (k >> 3)) & 1;
      const int q = NCB >= 2 ? 2 * ((p >> 1) ^ h) + (p & 1) : p;
      lds_direct_load16(W + ((int64_t)k * Cout + n0 + q * E::per_vec) * E::bytes,
                        (SHC_LDS void*)(wl + c * 1024));
    }
  } else {
    load_w(0, wv);
  }

  if constexpr (MODE == kPlanned) {
    // the row group's index lists, sort and job lists: the plan's image of
    // this LDS region, 64 vectors of 16 bytes per wavefront instruction (the
    // image is padded to whole 1 KB runs in the plan)
    const int ivecs = (ws_idx_bytes(R, K, kWaves, kRPT) + 1023) / 1024 * 64;
    const unsigned char* img = static_cast<const unsigned char*>(a.plan) +
                               (int64_t)blockIdx.x * a.plan_stride;
    unsigned char* ldst = smem + wbytes;
    for (int c = wave; c < ivecs / 64; c += kWaves)
      lds_direct_load16(img + (int64_t)c * 1024 + lane * 16, (SHC_LDS void*)(ldst + c * 1024));
  } else {
    for (int q = tid; q < R / 16; q += kThreads) blkmask[q] = 0;
    for (int q = tid; q < kBuckets; q += kThreads) bcnt[q] = 0;  // the sort's histogram
  }
  if constexpr (MODE != kPlanOut) {
    for (int q = tid; q < E::kstep * WROWW / 16; q += kThreads)
      reinterpret_cast<i32x4*>(zrows)[q] = i32x4{0, 0, 0, 0};
  }

  // ---- index lists, sorted by first sparse slot ---------------------------------
  // thread tid handles rows t = tid + rr * kThreads (rr < kRPT) of this workgroup
  if constexpr (MODE == kPlanned) {
    // from the plan (loaded above)
  } else if (CONV) {
    int32_t sv[kRPT][KM];
    if (TBL) {
      // one round: slot-major table rows, coalesced across the wavefront
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr) {
        const int t = tid + rr * kThreads;
        const int64_t i = row0 + (t < nrows ? t : nrows - 1);
#pragma unroll
        for (int j = 0; j < KM; ++j)
          sv[rr][j] = a.table[(int64_t)(j < K ? j : K - 1) * a.n_rows + i];
      }
      if constexpr (!DW) {
        store_w(0, wv);
        load_w(kWBatch * kThreads, wv);  // possibly all dummies: kept unconditional
      }
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr)
#pragma unroll
        for (int j = 0; j < KM; ++j)
          if (j >= K || tid + rr * kThreads >= nrows) sv[rr][j] = -1;
      if constexpr (!DW) store_w(kWBatch * kThreads, wv);
    } else {
      int rb[kRPT], rv[kRPT];
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr) {
        const int t = tid + rr * kThreads;
        const bool in = t < nrows;
        const int2 c = reinterpret_cast<const int2*>(a.coords)[row0 + (in ? t : 0)];
        const bool ok = in && c.x >= 0 && c.x < a.B && c.y >= 0 && c.y < a.V;
        rb[rr] = ok ? c.x : -1;
        rv[rr] = ok ? c.y : -1;
      }
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr)
#pragma unroll
        for (int j = 0; j < KM; ++j)
          sv[rr][j] = a.nbr[(int64_t)(rv[rr] >= 0 ? rv[rr] : 0) * K + (j < K ? j : K - 1)];
      store_w(0, wv);
      load_w(kWBatch * kThreads, wv);  // possibly all dummies: kept unconditional
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr)
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          const int32_t nb = sv[rr][j];
          sv[rr][j] = (j < K && rv[rr] >= 0 && nb >= 0 && nb < a.V) ? nb : -1;
        }
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr)
#pragma unroll
        for (int j = 0; j < KM; ++j) {
          const int32_t nb = sv[rr][j];
          sv[rr][j] = a.inv[(int64_t)(rb[rr] >= 0 ? rb[rr] : 0) * a.V + (nb >= 0 ? nb : 0)] |
                      (nb >= 0 ? 0 : int32_t(0x80000000));
        }
      store_w(kWBatch * kThreads, wv);
    }
    uint32_t rmask[kRPT];
#pragma unroll
    for (int rr = 0; rr < kRPT; ++rr) {
      rmask[rr] = 0;
#pragma unroll
      for (int j = 0; j < KM; ++j) {
        const int32_t s = sv[rr][j];
        sv[rr][j] = (uint32_t)s < (uint32_t)a.n_rows ? s : -1;  // 0 <= s < n_rows
        if (sv[rr][j] >= 0) rmask[rr] |= 1u << j;
      }
    }
    // weight vectors past the first two batches (large slices only)
    if constexpr (!DW) {
      for (int base = 2 * kWBatch * kThreads; base < wvecs; base += kWBatch * kThreads) {
        load_w(base, wv);
        store_w(base, wv);
      }
    }
    // rows per slot, then the dense slots
    for (int j = 0; j < K; ++j) {
      int c = 0;
#pragma unroll
      for (int rr = 0; rr < kRPT; ++rr) c += __popcll(__ballot((rmask[rr] >> j) & 1u));
      if (lane == 0) scnt[wave * kMaxSlots + j] = c;
    }
    __syncthreads();
    // dense slots (present in at least half of the rows): lane j of wave 0
    // sums slot j over the wavefronts, the mask goes out through LDS
    if (wave == 0) {
      int c = 0;
      if (lane < K)
        for (int w = 0; w < kWaves; ++w) c += scnt[w * kMaxSlots + lane];
      const uint64_t d = __ballot(lane < K && 2 * c >= nrows);
      if (lane == 0) scnt[kMaxSlots - 1] = (int32_t)(uint32_t)d;  // slot row of wave 0, K < kMaxSlots
    }
    __syncthreads();
    const uint32_t dense = (uint32_t)scnt[kMaxSlots - 1];
    // buckets: 0 = dense slots only, 1 + j = first sparse slot j, K + 1 = past
    // the end, -1 = no such row (t >= R).  A histogram (LDS atomics), its
    // exclusive scan, then a position per row from its bucket's cursor; the
    // order inside a bucket is whatever the atomics give, which no result
    // depends on (see the header).
    int* hist = bcnt;  // [kBuckets]: counts, then cursors
    int bkt[kRPT];
#pragma unroll
    for (int rr = 0; rr < kRPT; ++rr) {
      const int t = tid + rr * kThreads;
      const uint32_t key = rmask[rr] & ~dense;
      bkt[rr] = t >= R ? -1 : (t >= nrows ? K + 1 : (key ? 1 + __builtin_ctz(key) : 0));
      if (bkt[rr] >= 0) atomicAdd(&hist[bkt[rr]], 1);
    }
    __syncthreads();
    if (wave == 0) {  // exclusive scan of the K + 2 <= 34 counts, one per lane
      const int c = lane < K + 2 ? hist[lane] : 0;
      int inc = c;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(inc, d, 64);
        if (lane >= d) inc += y;
      }
      if (lane < K + 2) hist[lane] = inc - c;
    }
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < kRPT; ++rr) {
      if (bkt[rr] >= 0) {
        const int pos = atomicAdd(&hist[bkt[rr]], 1);
        perm[pos] = tid + rr * kThreads;
#pragma unroll
        for (int j = 0; j < KM; ++j)
          if (j < K) srcs[pos * K + j] = sv[rr][j];
        if (rmask[rr]) atomicOr(&blkmask[pos >> 4], rmask[rr]);
      }
    }
  } else {
    // input rows: row i itself, or (gather) row b_i * V + v_i of the dense
    // tensor; the coordinate loads go out with the weight slice's, before
    // either is used
    int2 cr[kRPT];
#pragma unroll
    for (int rr = 0; rr < kRPT; ++rr) {
      const int t = tid + rr * kThreads;
      cr[rr] = a.gather ? reinterpret_cast<const int2*>(a.coords)[row0 + (t < nrows ? t : 0)]
                        : int2{0, 0};
    }
    if constexpr (!DW) {
      for (int base = 0; base < wvecs; base += kWBatch * kThreads) {
        if (base > 0) load_w(base, wv);
        store_w(base, wv);
      }
    }
#pragma unroll
    for (int rr = 0; rr < kRPT; ++rr) {
      const int t = tid + rr * kThreads;
      if (t < R) {
        const int2 c = cr[rr];
        const bool ok = c.x >= 0 && c.x < a.B && c.y >= 0 && c.y < a.V;
        srcs[t] = t >= nrows ? -1 : (!a.gather ? (int32_t)(row0 + t) : (ok ? c.x * a.V + c.y : -1));
        perm[t] = t;
      }
    }
    for (int q = tid; q < R / 16; q += kThreads) blkmask[q] = (16 * q < nrows) ? 1u : 0u;
  }
  if constexpr (DW) __builtin_amdgcn_s_waitcnt(0);  // this wavefront's direct loads are in LDS
  __syncthreads();

  // ---- per-wave job loop -----------------------------------------------------------
  float bias_v[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int col = n0 + cb * 16 + l16;
    bias_v[cb] = (a.bias != nullptr && col < Cout) ? bias_raw[cb] : 0.f;
  }
  const bool relu = a.relu != 0;
  unsigned char* my_scratch = scratch + wave * 16 * WROW;

  struct Job {
    int blk;    // block, or -1 past the end
    int j;      // slot, or -1 for a block with no present slot (bias only)
    bool last;  // last job of its block
  };
  // This wavefront's job list, built once: its blocks b = wave, wave + 8, ...
  // in order, each with one job per live slot (ascending) or a single
  // bias-only job; packed as b << 8 | (slot + 1) << 1 | last.
  int njobs = 0;
  if constexpr (MODE == kPlanned) {
    // the plan's job count of this wavefront (at most kMaxJobs: a plan that
    // is not this shape's cannot run the loop past its list)
    njobs = min(scnt[wave], kMaxJobs);
  } else {
    const int nb = nblk > wave ? (nblk - wave + kWaves - 1) / kWaves : 0;
    int32_t* mine = jobl + wave * kMaxJobs;
    for (int i0 = 0; i0 < nb; i0 += 64) {
      const int i = i0 + lane;
      const int b = wave + kWaves * (i < nb ? i : 0);
      const uint32_t m = blkmask[b];
      const int c = i < nb ? (m ? __popc(m) : 1) : 0;
      int inc = c;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(inc, d, 64);
        if (lane >= d) inc += y;
      }
      int k = njobs + inc - c;
      if (i < nb) {
        if (m == 0) {
          mine[k] = (b << 8) | 1;
        } else {
          for (uint32_t mm = m; mm != 0;) {
            const int j = __builtin_ctz(mm);
            mm &= mm - 1;
            mine[k++] = (b << 8) | ((j + 1) << 1) | (mm == 0 ? 1 : 0);
          }
        }
      }
      njobs += __shfl(inc, 63, 64);
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  njobs = __builtin_amdgcn_readfirstlane(njobs);
  if constexpr (MODE == kPlanOut) {
    // every wavefront's job count beside its list (scnt is free after the
    // sort), then the whole region -- index lists, positions, block masks,
    // job lists -- to this row group's plan image
    if (lane == 0) scnt[wave] = njobs;
    __syncthreads();
    const int ibytes = ws_idx_bytes(R, K, kWaves, kRPT);
    const unsigned char* src = smem + wbytes;
    unsigned char* img = static_cast<unsigned char*>(a.plan_out) +
                         (int64_t)blockIdx.x * a.plan_stride;
    for (int q = tid; q < ibytes / 16; q += kThreads)
      *reinterpret_cast<i32x4*>(img + q * 16) = *reinterpret_cast<const i32x4*>(src + q * 16);
    return;
  }
  // lane l holds job (jt & ~63) + l; refilled every 64 jobs
  int jt = 0;
  int jreg = jobl[wave * kMaxJobs + lane];
  auto next_job = [&]() -> Job {
    if (jt >= njobs) return Job{-1, -1, true};
    if ((jt & 63) == 0 && jt > 0) jreg = jobl[wave * kMaxJobs + ((jt + lane) & (kMaxJobs - 1))];
    const int w = __builtin_amdgcn_readlane(jreg, jt & 63);
    ++jt;
    if (MODE == kPlanned && ((w >> 8) >= nblk || (w >> 8) < 0 || ((w >> 1) & 127) > K))
      return Job{-1, -1, true};
    return Job{w >> 8, ((w >> 1) & 127) - 1, (w & 1) != 0};
  };

  // A fragments come through raw buffer loads with 32-bit offsets: an absent
  // row (or a k-step past Cin) gets an offset beyond the buffer, and the
  // hardware returns zeros without touching memory.
  const int64_t s_rows = a.gather ? (int64_t)a.B * a.V : a.n_rows;  // rows of the input
  const __amdgpu_buffer_rsrc_t s_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.S), (short)0, (int)(s_rows * Cin * E::bytes), kBufferWord3);
  const uint32_t row_bytes = (uint32_t)Cin * E::bytes;
  struct Frags {
    i32x4 v[KSM];
  };
  auto issue = [&](const Job& jb, Frags& f) {
    const bool live = jb.blk >= 0 && jb.j >= 0;
    const int32_t src = live ? srcs[(jb.blk * 16 + l16) * K + jb.j] : -1;
    const uint32_t off = src >= 0 ? (uint32_t)src * row_bytes + (uint32_t)g * 16u : kOutOfRange;
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks)
      f.v[ks] = __builtin_bit_cast(
          i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     s_rsrc, ks < KS ? off + (uint32_t)ks * 64u : kOutOfRange, 0, 0));
  };

  // accumulators start at the bias of their column (lane l16 of block cb)
  f32x4 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = f32x4{bias_v[cb], bias_v[cb], bias_v[cb], bias_v[cb]};

  // B fragments of one k-step row block (bf16): two transposing LDS reads per
  // 16 output columns give lane (g, i) rows 8g .. 8g+7 of column i.
  auto read_b = [&](const unsigned char* base, bf16x8* out_cb) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const unsigned char* p0 =
          base + (8 * g + (l16 >> 2)) * WROWW + (((cb ^ swz_lane) << 5) + 8 * (l16 & 3));
      const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0)));
      const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0 + 4 * WROWW)));
      out_cb[cb] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
  };
  // The linear layer (one slot) multiplies every job by the same weights: a
  // wavefront keeps their B fragments in registers for the whole loop.
  constexpr bool kResidentB = BF16 && !CONV && KSM * NCB <= 32;  // at most 128 VGPRs
  bf16x8 wres[kResidentB ? KSM : 1][kResidentB ? NCB : 1];

  // Branch-free contraction of one job: every B fragment of the job is read
  // from LDS before the first MFMA (the scheduling barrier keeps the reads
  // ahead); a k-step past Cin reads the zero rows.
  auto compute = [&](const Job& jb, const Frags& f) {
    if (jb.blk < 0 || jb.j < 0) return;
    if (BF16) {
      if constexpr (kResidentB) {
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          const bf16x8 afrag = __builtin_bit_cast(bf16x8, f.v[ks]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb)
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                afrag, wres[kResidentB ? ks : 0][kResidentB ? cb : 0], acc[cb], 0, 0, 0);
        }
        return;
      }
      auto kbase = [&](int ks) {
        return ks < KS ? wl + (jb.j * Cin + ks * E::kstep) * WROWW : zrows;
      };
      if constexpr (KSM * NCB <= 8) {  // all of the job's B fragments: <= 32 VGPRs
        bf16x8 bfr[KSM][NCB];
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) read_b(kbase(ks), bfr[ks]);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          const bf16x8 afrag = __builtin_bit_cast(bf16x8, f.v[ks]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb)
            acc[cb] =
                __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag, bfr[ks][cb], acc[cb], 0, 0, 0);
        }
      } else {  // wide slices: read one k-step ahead
        bf16x8 bfr[2][NCB];
        read_b(kbase(0), bfr[0]);
#pragma unroll
        for (int ks = 0; ks < KSM; ++ks) {
          if (ks + 1 < KSM) read_b(kbase(ks + 1), bfr[(ks + 1) & 1]);
          __builtin_amdgcn_sched_barrier(0);
          const bf16x8 afrag = __builtin_bit_cast(bf16x8, f.v[ks]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb)
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag, bfr[ks & 1][cb], acc[cb],
                                                              0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    } else {
      // lane group g holds k = 4g .. 4g+3 of the k-step; MFMA s uses
      // component s of the A vector and slice row 4g + s
#pragma unroll
      for (int ks = 0; ks < KSM; ++ks) {
        const unsigned char* base =
            ks < KS ? wl + (jb.j * Cin + ks * E::kstep) * WROWW : zrows;
        float bw[NCB][4];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int s2 = 0; s2 < 4; ++s2)
            bw[cb][s2] = *reinterpret_cast<const float*>(base + (4 * g + s2) * WROWW +
                                                         (cb * 16 + l16) * 4);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int s2 = 0; s2 < 4; ++s2)
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(f.v[ks][s2]),
                                                           bw[cb][s2], acc[cb], 0, 0, 0);
      }
    }
  };

  // Output rows through raw buffer stores: positions past the rows of the
  // group (or columns past Cout) get an offset beyond the buffer and are dropped.
  const __amdgpu_buffer_rsrc_t o_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      a.out, (short)0, (int)(a.n_rows * Cout * E::bytes), kBufferWord3);
  auto epilogue = [&](int blk) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[cb][r];
        const float rx = x > 0.f ? x : 0.f;  // selects, no branch
        v[r] = relu ? rx : x;
      }
      unsigned char* pp = my_scratch + (g * 4) * WROW + (cb * 16 + l16) * E::bytes;
      if (BF16) {  // hardware round-to-nearest-even conversion, two rows per instruction
#pragma unroll
        for (int r = 0; r < 4; r += 2) {
          const bf16x2 h = __builtin_convertvector(f32x2{v[r], v[r + 1]}, bf16x2);
          *reinterpret_cast<__bf16*>(pp + r * WROW) = h[0];
          *reinterpret_cast<__bf16*>(pp + (r + 1) * WROW) = h[1];
        }
      } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) *reinterpret_cast<float*>(pp + r * WROW) = v[r];
      }
      acc[cb] = f32x4{bias_v[cb], bias_v[cb], bias_v[cb], bias_v[cb]};
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // every LDS read of the stores first (row positions, then the staged
    // vectors), then the stores: two LDS round trips, not one per store
    constexpr int NST = (16 * VPR + 63) / 64;
    int prow[NST];
    i32x4 sv[NST];
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int idx = t * 64 + lane;
      const int pos = blk * 16 + ((idx / VPR) & 15);
      prow[t] = perm[pos < nrows ? pos : 0];
    }
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int idx = t * 64 + lane;
      sv[t] = *reinterpret_cast<const i32x4*>(my_scratch + ((idx / VPR) & 15) * WROW +
                                              (idx % VPR) * 16);
    }
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int idx = t * 64 + lane;
      const int pos = blk * 16 + ((idx / VPR) & 15);
      const int n = n0 + (idx % VPR) * E::per_vec;
      const bool ok = idx < 16 * VPR && pos < nrows && n < Cout;
      const uint32_t off =
          ok ? ((uint32_t)(row0 + prow[t]) * (uint32_t)Cout + (uint32_t)n) * E::bytes
             : kOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u32, sv[t]), o_rsrc, off, 0, 0);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  // ring of D jobs; every slot of the ring issues its loads unconditionally
  Job jobs[D];
  Frags fr[D];
#pragma unroll
  for (int u = 0; u < D; ++u) {
    jobs[u] = next_job();
    issue(jobs[u], fr[u]);
  }
  // the resident B fragments are read once the first A loads are in flight
  if constexpr (kResidentB) {
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks)
      read_b(ks < KS ? wl + ks * E::kstep * WROWW : zrows, wres[kResidentB ? ks : 0]);
  }
  // Every ring slot is processed on every trip (an exhausted job computes
  // nothing and reloads a dummy address), so the loads of the other D - 1
  // jobs are never under a branch and stay in flight while one computes.
  while (jobs[0].blk >= 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      compute(jobs[u], fr[u]);
      if (jobs[u].blk >= 0 && jobs[u].last) epilogue(jobs[u].blk);
      jobs[u] = next_job();
      issue(jobs[u], fr[u]);
    }
  }
}

template <bool BF16, int WS, bool CONV, bool TBL, int KM, int KSM, bool DW = false,
          int MODE = kFull>
hipError_t launch_ws(const GemmArgs& a, const WsPlan& pl, hipStream_t stream) {
  const unsigned gx = (unsigned)((a.n_rows + pl.rows - 1) / pl.rows);
  // a plan is one image per row group, shared by the column slices
  const unsigned gy = MODE == kPlanOut ? 1u : (unsigned)((a.Cout + WS - 1) / WS);
  auto kern = ws_kernel<BF16, WS, CONV, TBL, KM, KSM, DW, MODE>;
  // allow the large dynamic LDS allocation; once per instantiation
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [&] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, kLdsLimit);
  });
  if (attr_err != hipSuccess) return attr_err;
  // a plan build holds only the index region in LDS
  const size_t lds = MODE == kPlanOut ? (size_t)pl.idx_bytes : (size_t)pl.total;
  hipLaunchKernelGGL(kern, dim3(gx, gy), dim3(CONV ? kThreadsConv : kThreadsLin), lds, stream, a,
                     pl.rows);
  return hipGetLastError();
}

template <bool BF16, int WS, bool CONV>
hipError_t launch_ws_k(const GemmArgs& a, const WsPlan& pl, hipStream_t stream) {
  constexpr int kstep = BF16 ? 32 : 16;
  const int ks = a.Cin / kstep;
  if (!CONV) {
    // direct weight loads: full column slices, whole 64-vector chunks
    const bool dw = BF16 && a.Cout % WS == 0 && ((int64_t)a.Cin * (WS * 2 / 16)) % 64 == 0;
    if (ks <= 4)
      return dw ? launch_ws<BF16, WS, false, false, 1, 4, BF16>(a, pl, stream)
                : launch_ws<BF16, WS, false, false, 1, 4>(a, pl, stream);
    return dw ? launch_ws<BF16, WS, false, false, 1, 8, BF16>(a, pl, stream)
              : launch_ws<BF16, WS, false, false, 1, 8>(a, pl, stream);
  }
  if (a.table != nullptr || a.plan != nullptr) {
    // direct weight loads: full column slices, whole 64-vector chunks
    const bool dw = BF16 && a.Cout % WS == 0 && ((int64_t)a.K * a.Cin * (WS * 2 / 16)) % 64 == 0;
    if constexpr (BF16) {
      if (dw && a.plan_out != nullptr)
        return ks <= 4 ? launch_ws<true, WS, true, true, 10, 4, true, kPlanOut>(a, pl, stream)
                       : launch_ws<true, WS, true, true, 10, 8, true, kPlanOut>(a, pl, stream);
      if (dw && a.plan != nullptr)
        return ks <= 4 ? launch_ws<true, WS, true, true, 10, 4, true, kPlanned>(a, pl, stream)
                       : launch_ws<true, WS, true, true, 10, 8, true, kPlanned>(a, pl, stream);
    }
    if (a.plan_out != nullptr || a.table == nullptr) return hipErrorInvalidValue;
    if (ks <= 4)
      return dw ? launch_ws<BF16, WS, true, true, 10, 4, BF16>(a, pl, stream)
                : launch_ws<BF16, WS, true, true, 10, 4>(a, pl, stream);
    return dw ? launch_ws<BF16, WS, true, true, 10, 8, BF16>(a, pl, stream)
              : launch_ws<BF16, WS, true, true, 10, 8>(a, pl, stream);
  }
  if (ks <= 4) return launch_ws<BF16, WS, true, false, 10, 4>(a, pl, stream);
  return launch_ws<BF16, WS, true, false, 10, 8>(a, pl, stream);
}

}  // namespace

// Plan for the weight-stationary kernel, or false when the shape does not fit.
bool ws_plan(const GemmArgs& a, bool conv, bool bf16, int num_cus, WsPlan* pl) {
  const int nt = conv ? kThreadsConv : kThreadsLin;
  const int waves = nt / 64, rpt = kMaxRows / nt;
  const int e = bf16 ? 2 : 4;
  const int K = conv ? a.K : 1;
  const int Ktot = K * a.Cin;
  const int kstep = bf16 ? 32 : 16;
  if ((a.Cin * e) % 64 != 0) return false;  // whole 64-byte k-steps per slot
  if (a.Cin / kstep > 8) return false;       // at most 8 k-steps per slot job
  if (conv && K > 10) return false;          // index build keeps <= 10 slots per row
  // 32-bit buffer offsets, with kOutOfRange past the end of every buffer
  if ((a.gather ? (int64_t)a.B * a.V : a.n_rows) * a.Cin * e > 0x7FFF0000LL) return false;
  if ((int64_t)a.n_rows * a.Cout * e > 0x7FFF0000LL) return false;
  // sparse inputs only: at high density the tiled kernel (gemm.hip) is faster
  // than building the index lists here (with a prebuilt table there is none)
  if (conv && a.table == nullptr && a.plan == nullptr && a.plan_out == nullptr &&
      (double)a.n_rows > 0.3 * (double)a.B * (double)a.V)
    return false;
  int ws = 0;
  for (int cand : {128, 64, 32}) {
    if (cand > ((a.Cout + 15) / 16) * 16 && cand != 32) continue;
    const int wb = ((Ktot * ws_wrow_w(cand, e) + 15) & ~15);
    if (wb + ws_scratch(cand, e, waves) + ws_idx_bytes(256, K, waves, rpt) <= kLdsLimit) {
      ws = cand;
      break;
    }
  }
  if (ws == 0) return false;
  const int slices = (a.Cout + ws - 1) / ws;
  const int wb = (Ktot * ws_wrow_w(ws, e) + 15) & ~15;
  // rows per workgroup: one workgroup per CU when the rows fit, within LDS
  int64_t target = (a.n_rows * slices + num_cus - 1) / num_cus;
  // Beyond one wave of workgroups the tiled kernel is faster for the conv
  // (measured: 20% active rows of a 1.34M-row batch at C = 128 take 141 us
  // tiled against 194 us here); the weight slice and sorting are per workgroup.
  if (conv && target > kMaxRows) return false;
  int rows = (int)((target + 15) / 16) * 16;
  if (rows < 64) rows = 64;
  if (rows > kMaxRows) rows = kMaxRows;
  while (rows > 64 && wb + ws_scratch(ws, e, waves) + ws_idx_bytes(rows, K, waves, rpt) > kLdsLimit) rows -= 16;
  if (wb + ws_scratch(ws, e, waves) + ws_idx_bytes(rows, K, waves, rpt) > kLdsLimit) return false;
  pl->ws = ws;
  pl->wrow = ws_wrow_w(ws, e);
  pl->wbytes = wb;
  pl->rows = rows;
  pl->idx_bytes = ws_idx_bytes(rows, K, waves, rpt);
  pl->scratch = ws_scratch(ws, e, waves);
  pl->total = wb + pl->idx_bytes + pl->scratch;
  return true;
}

int64_t conv_plan_bytes(const GemmArgs& a_in, bool bf16, int num_cus, int64_t* stride) {
  *stride = 0;
  // sized as the conv from a table that builds it (the pointer is never read)
  GemmArgs a = a_in;
  a.plan_out = &a;
  WsPlan pl;
  if (!bf16 || a.n_rows <= 0 || !ws_plan(a, true, true, num_cus, &pl)) return 0;
  // the same condition as the launch's direct weight loads
  if (a.Cout % pl.ws != 0 || ((int64_t)a.K * a.Cin * (pl.ws * 2 / 16)) % 64 != 0) return 0;
  const int waves = kThreadsConv / 64, rpt = kMaxRows / kThreadsConv;
  *stride = ((int64_t)ws_idx_bytes(pl.rows, a.K, waves, rpt) + 1023) / 1024 * 1024;
  return ((a.n_rows + pl.rows - 1) / pl.rows) * *stride;
}

int64_t conv_plan_max_rows(const GemmArgs& a_in, bool bf16, int num_cus) {
  // A plan exists for every row count up to a limit (the one-wave and 32-bit
  // offset bounds of ws_plan grow with n, the rest does not depend on it).
  GemmArgs a = a_in;
  int64_t st;
  a.n_rows = 1;
  if (conv_plan_bytes(a, bf16, num_cus, &st) == 0) return 0;
  int64_t lo = 1, hi = INT32_MAX;  // plan at lo; find the last n with one
  a.n_rows = hi;
  if (conv_plan_bytes(a, bf16, num_cus, &st) > 0) return hi;
  while (hi - lo > 1) {
    const int64_t mid = lo + (hi - lo) / 2;
    a.n_rows = mid;
    if (conv_plan_bytes(a, bf16, num_cus, &st) > 0) lo = mid; else hi = mid;
  }
  return lo;
}

int64_t conv_plan_bytes_upto(const GemmArgs& a_in, bool bf16, int num_cus) {
  // Rows per group R(n) rise in steps of 16 with n, and within a step the plan
  // (row groups x image stride) only grows; so the largest plan of any n <=
  // n_rows is at the end of a step or at the last n that takes a plan.
  const int64_t nmax = std::min<int64_t>(a_in.n_rows, conv_plan_max_rows(a_in, bf16, num_cus));
  if (nmax <= 0) return 0;
  GemmArgs a = a_in;
  a.n_rows = 1;
  a.plan_out = &a;
  WsPlan pl;
  if (!ws_plan(a, true, true, num_cus, &pl)) return 0;
  const int64_t slices = (a.Cout + pl.ws - 1) / pl.ws;
  int64_t best = 0, st;
  for (int r = 64; r <= kMaxRows + 16; r += 16) {
    const int64_t n = r > kMaxRows ? nmax : std::min(nmax, (int64_t)r * num_cus / slices);
    if (n <= 0) continue;
    a.n_rows = n;
    best = std::max(best, conv_plan_bytes(a, bf16, num_cus, &st));
  }
  return best;
}

hipError_t launch_ws_gemm(const GemmArgs& a, bool conv, bool bf16, const WsPlan& pl,
                          hipStream_t stream) {
#define SHC_WS_CASE(BF, WSV)                                                               \
  if (pl.ws == WSV)                                                                        \
    return conv ? launch_ws_k<BF, WSV, true>(a, pl, stream)                                \
                : launch_ws_k<BF, WSV, false>(a, pl, stream);
  if (bf16) {
    SHC_WS_CASE(true, 128) SHC_WS_CASE(true, 64) SHC_WS_CASE(true, 32)
  } else {
    SHC_WS_CASE(false, 128) SHC_WS_CASE(false, 64) SHC_WS_CASE(false, 32)
  }
#undef SHC_WS_CASE
  return hipErrorInvalidValue;
}

}  // namespace shc
