// Sparse neighbourhood convolution from a neighbour-row table (Eqs. 4-5,
// with the activation of Eq. 10), bf16, with slot 0 and the other slots
// computed apart:
//
//   out[i] = act( bias + sum_{1 <= j < K} P[j][i] + S[table[0][i]] W[0] ),
//   P[j][i] = S[table[j][i]] W[j]   where table[j][i] >= 0 (else no term).
//
// Slot 0 of a spiral or k-NN neighbourhood is the vertex itself, present in
// every row; under a sparse mask the other slots are mostly absent (at 10%
// density about one row in ten has a given one).  Two launches:
//
//   pair launch: a workgroup owns one slot j >= 1 and a chunk of rows.  It
//     holds W[j] (every output column) in LDS, lists the chunk's rows whose
//     slot j is present, and multiplies their neighbour rows by W[j] in jobs
//     of 16 (row, slot) pairs, writing each P[j][i] in fp32 to a workspace
//     [K - 1][n_rows][Cout] (absent pairs are neither written nor read);
//   row launch: a workgroup holds W[0] in LDS and its wavefronts walk groups
//     of rows.  A row's accumulators start at its first present P[j][i] plus
//     the bias, then take its other present P[j][i] in slot order, and the
//     slot-0 product is accumulated onto them on the matrix cores; then the
//     activation and the rounding to bf16.
//
// Every weight matrix reaches a CU once per workgroup and every gathered
// neighbour row once for all output columns, where the tiled kernel re-reads
// the weights per 128-row tile and the weight-stationary one the rows per
// column slice.  The price is the fp32 round trip of the present pairs'
// partial rows through the workspace, so the split pays at low density and
// wide rows.  The order of the sums is fixed (the present slots j >= 1
// ascending, with the bias added after the first, then slot 0's k-steps), so
// the result does not depend on how rows or pairs are spread over
// workgroups.
//
// MFMAs run transposed (D^T = W^T S^T): the A operand is a 16-column block of
// W read with the transposing LDS load, the B operand 16 gathered rows of S
// (16 contiguous bytes per lane), and lane (g, i) of the 16 x 16 result holds
// output columns 4g .. 4g+3 of row i: 16 contiguous fp32 bytes of a partial
// row, or 8 of an output row, per lane and column block.
#include <hip/hip_runtime.h>

#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kSpLdsLimit = 160 * 1024;
constexpr int kSpBufferWord3 = 0x00020000;  // raw buffer resource, 32-bit data
constexpr uint32_t kSpOutOfRange = 0x80000000u;
constexpr int kPairThreads = 256;
constexpr int kPairLoads = 24;                               // table loads per thread
constexpr int kMaxChunkRows = kPairLoads * kPairThreads;     // one pass over a chunk
static_assert(kMaxChunkRows <= 65536, "chunk rows fit the 16-bit pair lists");
#define SHC_SP_LDS __attribute__((address_space(3)))

typedef __bf16 sp_bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef __bf16 sp_bf16x2 __attribute__((ext_vector_type(2)));
typedef float sp_f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t sp_v4u32 __attribute__((ext_vector_type(4)));
typedef uint32_t sp_v2u32 __attribute__((ext_vector_type(2)));

struct SplitArgs {
  const void* S;         // [n_rows][Cin] bf16
  const int32_t* table;  // [K][n_rows]
  const void* W;         // [K][Cin][Cout] bf16
  const float* bias;     // [Cout] or null
  void* out;             // [n_rows][Cout] bf16
  float* P;              // [K - 1][n_rows][Cout] fp32
  int64_t n_rows;
  int32_t K;
  int32_t relu;
  int32_t chunk_rows;    // pair launch: rows per workgroup
};

// A workgroup barrier that orders LDS only (global loads stay in flight).
__device__ __forceinline__ void sp_lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Weights of one slot in LDS, [Cin][Cout] bf16 rows of 2 Cout bytes whose
// 32-byte column chunk c sits at c ^ swz(r).  A transposing read touches
// rows 8g + i (+ 4) for g, i < 4, each half-wavefront 8 of them; with rows of
// 256 or 512 bytes every row starts on bank 0, and the three bits of the XOR
// put those 8 rows on 8 different bank groups; with 128-byte rows (two to a
// bank cycle) two bits do it.
template <int NCT>
__device__ __forceinline__ int sp_swz(int r) {
  if constexpr (NCT >= 8) return (r & 3) | (((r >> 3) & 1) << 2);
  else return ((r >> 1) & 1) | (((r >> 3) & 1) << 1);
}

template <int KS, int NCT, int NT>
struct SlotWeights {
  static constexpr int Cin = KS * 32;
  static constexpr int Cout = NCT * 16;
  static constexpr int WROW = Cout * 2;
  static constexpr int VPR = WROW / 16;
  static constexpr int VECS = Cin * VPR;  // 16-byte vectors
  static_assert(VECS % 64 == 0, "whole wavefront loads");
  static constexpr int bytes = Cin * WROW;

  // W[j] straight into LDS with 16-byte direct loads: LDS vector v (row
  // k = v / VPR, position p = v % VPR) receives source vector q of row k with
  // q's chunk swizzled to p's (the XOR is its own inverse).  A wavefront's
  // load writes 64 consecutive vectors; the caller waits for its own loads
  // (s_waitcnt) before the barrier that publishes them.
  __device__ static void load(const void* W, int j, int tid, unsigned char* wbuf,
                              int k0 = 0, int kr = Cin) {
    const unsigned char* src =
        static_cast<const unsigned char*>(W) + (int64_t)j * bytes + (int64_t)k0 * WROW;
    const int lane = tid & 63;
    for (int c = tid >> 6; c < kr * VPR / 64; c += NT / 64) {
      const int v = c * 64 + lane;
      const int k = v / VPR;
      const int p = v - k * VPR;
      const int q = 2 * ((p >> 1) ^ sp_swz<NCT>(k)) + (p & 1);
      __builtin_amdgcn_global_load_lds(src + (k * VPR + q) * 16,
                                       (SHC_SP_LDS void*)(wbuf + c * 1024), 16, 0, 0);
    }
  }
  // the A operand of k-step ks and column block ct: lane (g, i) gets W rows
  // 32 ks + 8g .. +7 of column 16 ct + i (two transposing reads)
  __device__ static bf16x8 read(const unsigned char* wbuf, int ks, int ct, int g, int l16) {
    const int swz = sp_swz<NCT>(8 * g + (l16 >> 2));
    const unsigned char* p0 = wbuf + (ks * 32 + 8 * g + (l16 >> 2)) * WROW + 8 * (l16 & 3) +
                              ((ct ^ swz) << 5);
    const sp_bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_SP_LDS sp_bf16x4*)(const_cast<unsigned char*>(p0)));
    const sp_bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_SP_LDS sp_bf16x4*)(const_cast<unsigned char*>(p0 + 4 * WROW)));
    return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
};

__device__ __forceinline__ int sp_lanes_below(uint64_t bal) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(bal >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)bal, 0u));
}

// ---------------------------------------------------------------------------
// pair launch: grid (chunks, K - 1), workgroup (chunk c, slot j = 1 + y).
// Wavefront w owns a quarter of the output columns: it reads its weight
// fragments of W[j] from LDS once, into registers, and then takes every job
// of the workgroup for those columns.  A job's 16 neighbour rows are staged
// in LDS once for the four wavefronts, kPairBatch jobs at a time and double
// buffered (the next batch's rows in flight in registers while one batch
// computes); the weights' LDS region holds the staging buffers once the
// fragments are in registers.
// ---------------------------------------------------------------------------
constexpr int kPairBatch = 4;  // jobs staged per barrier

__host__ __device__ constexpr int sp_stage_row(int cin) { return cin * 2 + 16; }
__host__ __device__ constexpr int sp_pair_region(int cin, int cout, int wp) {
  // a slice of the slot's weights, or two staging buffers of kPairBatch
  // jobs, the larger
  return cin * cout * 2 / wp > 2 * kPairBatch * 16 * sp_stage_row(cin)
             ? cin * cout * 2 / wp
             : 2 * kPairBatch * 16 * sp_stage_row(cin);
}

// (WP: parts the slot's weights are staged in, a slice of Cin / WP rows at a
// time, so that two workgroups fit a CU)
template <int KS, int NCT, int WP>
__global__ __launch_bounds__(kPairThreads, 2) void conv_pairs_kernel(const SplitArgs a) {
  constexpr int NT = kPairThreads;
  constexpr int NW = NT / 64;
  using SW = SlotWeights<KS, NCT, NT>;
  constexpr int Cin = SW::Cin;
  constexpr int Cout = SW::Cout;
  constexpr int NCTW = NCT / NW;                 // column blocks per wavefront
  static_assert(NCT % NW == 0, "whole column blocks per wavefront");
  constexpr int SROW = sp_stage_row(Cin);        // staged row, padded by 16 bytes
  constexpr int SBUF = kPairBatch * 16 * SROW;   // one staging buffer
  constexpr int VPRow = Cin * 2 / 16;            // 16-byte vectors per row
  constexpr int SV = kPairBatch * 16 * VPRow / NT;  // staged vectors per thread
  static_assert((kPairBatch * 16 * VPRow) % NT == 0, "whole staged vectors per thread");

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int rc = a.chunk_rows;
  unsigned char* region = smem;  // W[j], then the staging buffers
  // pair lists: neighbour rows, then the rows themselves relative to the
  // chunk (16 bits: rc <= kMaxChunkRows), then the count
  int32_t* srcl = reinterpret_cast<int32_t*>(smem + sp_pair_region(Cin, Cout, WP));  // [rc]
  uint16_t* dstl = reinterpret_cast<uint16_t*>(srcl + rc);                        // [rc]
  int32_t* cnt = reinterpret_cast<int32_t*>(dstl + ((rc + 1) & ~1));              // pairs

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 4;
  const int l16 = lane & 15;
  const int j = blockIdx.y + 1;
  const int64_t n = a.n_rows;
  const int64_t row0 = (int64_t)blockIdx.x * rc;
  const int nrows = (int)min((int64_t)rc, n - row0);

  static_assert(KS % WP == 0, "whole k-steps per slice of the weights");
  constexpr int KSP = KS / WP;  // k-steps per slice
  SW::load(a.W, j, tid, region, 0, KSP * 32);
  if (tid == 0) *cnt = 0;
  // the chunk's slot-j entries, all in flight at once (rc <= kMaxChunkRows)
  const int32_t* tj = a.table + (int64_t)j * n + row0;
  int32_t s[kPairLoads];
#pragma unroll
  for (int u = 0; u < kPairLoads; ++u) {
    const int t = u * NT + tid;
    s[u] = t < nrows ? tj[t] : -1;
  }
  __builtin_amdgcn_s_waitcnt(0);  // the direct weight loads and the entries are in
  sp_lds_barrier();

  // this wavefront's weight fragments, for good, slice by slice
  bf16x8 wreg[KS][NCTW];
#pragma unroll
  for (int wp = 0; wp < WP; ++wp) {
    if (wp > 0) {
      sp_lds_barrier();  // the previous slice's fragments are read
      SW::load(a.W, j, tid, region, wp * KSP * 32, KSP * 32);
      __builtin_amdgcn_s_waitcnt(0);
      sp_lds_barrier();
    }
#pragma unroll
    for (int ks = 0; ks < KSP; ++ks)
#pragma unroll
      for (int c = 0; c < NCTW; ++c)
        wreg[wp * KSP + ks][c] = SW::read(region, ks, wave * NCTW + c, g, l16);
  }

  // the present pairs (list order is immaterial: every pair's partial row is
  // computed on its own and stored by row): one LDS atomic per wavefront
  // reserves its pairs' places, the lanes' ballots place them
  uint64_t bal[kPairLoads];
  int total = 0;
#pragma unroll
  for (int u = 0; u < kPairLoads; ++u) {
    bal[u] = __ballot((uint32_t)s[u] < (uint32_t)n);  // rows past the chunk read -1
    total += (int)__popcll(bal[u]);
  }
  int base = 0;
  if (lane == 0 && total > 0) base = atomicAdd(cnt, total);
  base = __shfl(base, 0);
#pragma unroll
  for (int u = 0; u < kPairLoads; ++u) {
    if ((bal[u] >> lane) & 1) {
      const int pos = base + sp_lanes_below(bal[u]);
      srcl[pos] = s[u];
      dstl[pos] = (uint16_t)(u * NT + tid);
    }
    base += (int)__popcll(bal[u]);
  }
  // the lists are complete and every wavefront's fragments are read: the
  // weights' region becomes the staging buffers
  __builtin_amdgcn_s_waitcnt(0);
  sp_lds_barrier();
  const int np = *cnt;
  const int nb = (np + kPairBatch * 16 - 1) / (kPairBatch * 16);  // batches of jobs

  const __amdgpu_buffer_rsrc_t s_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.S), (short)0, (int)(n * Cin * 2), kSpBufferWord3);
  unsigned char* pj = reinterpret_cast<unsigned char*>(a.P) + (int64_t)(j - 1) * n * Cout * 4;
  const __amdgpu_buffer_rsrc_t p_rsrc =
      __builtin_amdgcn_make_buffer_rsrc(pj, (short)0, (int)(n * Cout * 4), kSpBufferWord3);

  // batch b: pairs kPairBatch * 16 * b + r, r < kPairBatch * 16; staged
  // vector v = u * NT + tid is row r = v / VPRow, 16 bytes c = v % VPRow
  // (an absent pair's row reads zeros)
  i32x4 sreg[SV];
  auto load_batch = [&](int b) {
#pragma unroll
    for (int u = 0; u < SV; ++u) {
      const int v = u * NT + tid;
      const int r = v / VPRow, c = v - (v / VPRow) * VPRow;
      const int p = b * kPairBatch * 16 + r;
      const int32_t src = p < np ? srcl[p] : -1;
      sreg[u] = __builtin_bit_cast(
          i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     s_rsrc,
                     src >= 0 ? (uint32_t)src * (uint32_t)(Cin * 2) + (uint32_t)c * 16u
                              : kSpOutOfRange,
                     0, 0));
    }
  };
  auto store_batch = [&](int buf) {
    unsigned char* dst = region + buf * SBUF;
#pragma unroll
    for (int u = 0; u < SV; ++u) {
      const int v = u * NT + tid;
      const int r = v / VPRow, c = v - (v / VPRow) * VPRow;
      *reinterpret_cast<i32x4*>(dst + r * SROW + c * 16) = sreg[u];
    }
  };
  auto compute_batch = [&](int b, int buf) {
    const unsigned char* rows = region + buf * SBUF;
#pragma unroll
    for (int jj = 0; jj < kPairBatch; ++jj) {
      // B operand of k-step ks: 16 bytes of staged row jj * 16 + i, k-group g
      const unsigned char* rp = rows + (jj * 16 + l16) * SROW + g * 16;
      f32x4 acc[NCTW];
#pragma unroll
      for (int c = 0; c < NCTW; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 sf = *reinterpret_cast<const bf16x8*>(rp + ks * 64);
#pragma unroll
        for (int c = 0; c < NCTW; ++c)
          acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wreg[ks][c], sf, acc[c], 0, 0, 0);
      }
      const int p = (b * kPairBatch + jj) * 16 + l16;
      const int32_t dst = p < np ? (int32_t)(row0 + dstl[p]) : -1;
      const uint32_t off = (uint32_t)dst * (uint32_t)(Cout * 4) +
                           (uint32_t)(wave * NCTW) * 64u + (uint32_t)g * 16u;
#pragma unroll
      for (int c = 0; c < NCTW; ++c)
        __builtin_amdgcn_raw_buffer_store_b128(
            __builtin_bit_cast(sp_v4u32, acc[c]), p_rsrc,
            dst >= 0 ? off + (uint32_t)c * 64u : kSpOutOfRange, 0, 0);
    }
  };

  if (nb > 0) {
    load_batch(0);
    store_batch(0);
    sp_lds_barrier();
  }
  for (int b = 0; b < nb; ++b) {
    if (b + 1 < nb) load_batch(b + 1);
    compute_batch(b, b & 1);
    if (b + 1 < nb) store_batch((b + 1) & 1);
    sp_lds_barrier();
  }
}

// ---------------------------------------------------------------------------
// row launch: four wavefronts per workgroup, wavefront w owning a quarter of
// the output columns with its weight fragments of W[0] in registers for the
// whole launch.  Workgroups walk batches of kRowBatch 16-row blocks,
// grid-stride; a batch's input rows are staged in LDS once for the four
// wavefronts (the next batch's rows and table entries in flight while one
// computes), each wavefront loads its own columns of the rows' partial rows.
// JQ table entries per lane and block (lane (g, i) reads slots g, g + 4, ...
// of row i).
// ---------------------------------------------------------------------------
constexpr int kRowBatch = 4;  // 16-row blocks per batch (two for big shapes)

__host__ __device__ constexpr int sp_row_region(int cin, int cout, int rb, int wp) {
  // a slice of W[0], or two staging buffers of a batch's rows, the larger
  return cin * cout * 2 / wp > 2 * rb * 16 * sp_stage_row(cin) ? cin * cout * 2 / wp
                                                               : 2 * rb * 16 * sp_stage_row(cin);
}

// RB: 16-row blocks per batch; WP: parts W[0] is staged in (its rows in WP
// slices of Cin / WP), so that the LDS a workgroup holds is the larger of a
// slice and the two staging buffers.
template <int KS, int NCT, int JQ, int MINW, int RB, int WP>
__global__ __launch_bounds__(kPairThreads, MINW) void conv_rows_kernel(const SplitArgs a) {
  constexpr int NT = kPairThreads;
  constexpr int NW = NT / 64;
  using SW = SlotWeights<KS, NCT, NT>;
  constexpr int Cin = SW::Cin;
  constexpr int Cout = SW::Cout;
  constexpr int NCTW = NCT / NW;
  static_assert(NCT % NW == 0, "whole column blocks per wavefront");
  static_assert(KS % WP == 0, "whole k-steps per slice of W[0]");
  constexpr int SROW = sp_stage_row(Cin);
  constexpr int SBUF = RB * 16 * SROW;
  constexpr int VPRow = Cin * 2 / 16;
  constexpr int SV = RB * 16 * VPRow / NT;  // staged vectors per thread
  static_assert((RB * 16 * VPRow) % NT == 0, "whole staged vectors per thread");

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* region = smem;  // W[0], then the staging buffers

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 4;
  const int l16 = lane & 15;
  const int64_t n = a.n_rows;
  const int K = a.K;
  const int64_t nbatch = (n + RB * 16 - 1) / (RB * 16);
  const int64_t stride = gridDim.x;

  const __amdgpu_buffer_rsrc_t s_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.S), (short)0, (int)(n * Cin * 2), kSpBufferWord3);
  const __amdgpu_buffer_rsrc_t p_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      a.P, (short)0, (int)((int64_t)(K > 1 ? K - 1 : 1) * n * Cout * 4), kSpBufferWord3);
  const __amdgpu_buffer_rsrc_t o_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      a.out, (short)0, (int)(n * Cout * 2), kSpBufferWord3);

  // this wavefront's weight fragments of W[0], for good, a slice of W[0]'s
  // rows at a time through LDS
  bf16x8 wreg[KS][NCTW];
#pragma unroll
  for (int wp = 0; wp < WP; ++wp) {
    constexpr int KSP = KS / WP;  // k-steps per slice
    SW::load(a.W, 0, tid, region, wp * KSP * 32, KSP * 32);
    __builtin_amdgcn_s_waitcnt(0);
    sp_lds_barrier();
#pragma unroll
    for (int ks = 0; ks < KSP; ++ks)
#pragma unroll
      for (int c = 0; c < NCTW; ++c)
        wreg[wp * KSP + ks][c] = SW::read(region, ks, wave * NCTW + c, g, l16);
    sp_lds_barrier();  // the slice's fragments are read: the region is free again
  }

  // A batch's table entries (this lane's row of each block) and input rows.
  // The rows are staged as each row's own input row, which is slot 0's
  // neighbour row in a spiral or k-NN table; a block whose table says
  // otherwise reads its slot-0 rows from memory instead.
  int32_t sv[RB][JQ];
  i32x4 sreg[SV];
  auto load_entries = [&](int64_t b) {
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      const int64_t row = (b * RB + u) * 16 + l16;
      const bool valid = row < n;
#pragma unroll
      for (int q = 0; q < JQ; ++q) {
        const int jq = g + 4 * q;
        const int jc = jq < K ? jq : K - 1;
        sv[u][q] = valid ? a.table[(int64_t)jc * n + row] : -1;
      }
    }
  };
  auto load_rows = [&](int64_t b) {
#pragma unroll
    for (int u = 0; u < SV; ++u) {
      const int v = u * NT + tid;
      const int r = v / VPRow, c = v - (v / VPRow) * VPRow;
      const int64_t row = b * RB * 16 + r;
      sreg[u] = __builtin_bit_cast(
          i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     s_rsrc,
                     row < n ? (uint32_t)row * (uint32_t)(Cin * 2) + (uint32_t)c * 16u
                             : kSpOutOfRange,
                     0, 0));
    }
  };
  auto store_rows = [&](int buf) {
    unsigned char* dst = region + buf * SBUF;
#pragma unroll
    for (int u = 0; u < SV; ++u) {
      const int v = u * NT + tid;
      const int r = v / VPRow, c = v - (v / VPRow) * VPRow;
      *reinterpret_cast<i32x4*>(dst + r * SROW + c * 16) = sreg[u];
    }
  };
  // this wavefront's columns of partial row P[j][r] (zeros for j = 0)
  auto load_p = [&](int j, int64_t r, f32x4 (&c)[NCTW]) {
    const uint32_t off = j > 0 ? ((uint32_t)(j - 1) * (uint32_t)n + (uint32_t)r) *
                                         (uint32_t)(Cout * 4) +
                                     (uint32_t)(wave * NCTW) * 64u + (uint32_t)g * 16u
                               : 0u;
#pragma unroll
    for (int q = 0; q < NCTW; ++q)
      c[q] = __builtin_bit_cast(
          f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     p_rsrc, j > 0 ? off + (uint32_t)q * 64u : kSpOutOfRange, 0, 0));
  };

  int64_t b = blockIdx.x;
  if (b < nbatch) {
    load_entries(b);
    load_rows(b);
    store_rows(0);
  }
  sp_lds_barrier();
  int buf = 0;
  const bool relu = a.relu != 0;
  for (; b < nbatch; b += stride) {
    // present-slot masks and slot-0 rows of the batch's blocks
    int64_t row[RB];
    uint32_t m[RB];
    int32_t s0[RB];
    bool staged[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      row[u] = (b * RB + u) * 16 + l16;
      m[u] = 0;
      s0[u] = -1;
#pragma unroll
      for (int q = 0; q < JQ; ++q) {
        const int jq = g + 4 * q;
        const bool ok = jq < K && (uint32_t)sv[u][q] < (uint32_t)n;
        m[u] |= (ok ? 1u : 0u) << jq;
        if (q == 0) s0[u] = ok ? sv[u][0] : -1;
      }
      m[u] |= (uint32_t)__shfl_xor((int)m[u], 16);
      m[u] |= (uint32_t)__shfl_xor((int)m[u], 32);
      s0[u] = __shfl(s0[u], l16);  // from lane (0, i)
      staged[u] = __ballot(row[u] < n && s0[u] != row[u]) == 0;
    }
    // accumulators: first present slot j >= 1's partial row, plus the bias,
    // plus the second one (loaded beside the first); then any further ones
    f32x4 acc[RB][NCTW], c2[RB][NCTW];
    uint32_t rest[RB];
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      const uint32_t sp = m[u] & ~1u;
      const uint32_t sp2 = sp & (sp - 1u);
      load_p(sp ? __builtin_ctz(sp) : 0, row[u], acc[u]);
      load_p(sp2 ? __builtin_ctz(sp2) : 0, row[u], c2[u]);
      rest[u] = sp2 & (sp2 - 1u);
    }
    // the next batch's entries and rows go out now
    const bool more = b + stride < nbatch;
    if (more) {
      load_entries(b + stride);
      load_rows(b + stride);
    }
#pragma unroll
    for (int q = 0; q < NCTW; ++q) {
      const int col = (wave * NCTW + q) * 16 + 4 * g;
      f32x4 bv = {0.f, 0.f, 0.f, 0.f};
      if (a.bias != nullptr)
        bv = f32x4{a.bias[col], a.bias[col + 1], a.bias[col + 2], a.bias[col + 3]};
#pragma unroll
      for (int u = 0; u < RB; ++u) acc[u][q] = (acc[u][q] + bv) + c2[u][q];
    }
    // (all blocks' next further slots in one round trip per round)
    uint32_t any = 0;
#pragma unroll
    for (int u = 0; u < RB; ++u) any |= rest[u];
    while (__ballot(any != 0) != 0) {
      f32x4 c[RB][NCTW];
#pragma unroll
      for (int u = 0; u < RB; ++u) load_p(rest[u] != 0 ? __builtin_ctz(rest[u]) : 0, row[u], c[u]);
      any = 0;
#pragma unroll
      for (int u = 0; u < RB; ++u) {
#pragma unroll
        for (int q = 0; q < NCTW; ++q) acc[u][q] += c[u][q];
        rest[u] &= rest[u] - 1u;
        any |= rest[u];
      }
    }

    // slot 0 on the matrix cores: B operands from the staged rows, or from
    // memory for a block whose slot 0 is not the row itself
    const unsigned char* rows = region + buf * SBUF;
#pragma unroll
    for (int u = 0; u < RB; ++u) {
      if (staged[u]) {
        // every k-step's B operand read first: the reads' latency is paid once
        const unsigned char* rp = rows + (u * 16 + l16) * SROW + g * 16;
        bf16x8 sf[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) sf[ks] = *reinterpret_cast<const bf16x8*>(rp + ks * 64);
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
#pragma unroll
          for (int q = 0; q < NCTW; ++q)
            acc[u][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wreg[ks][q], sf[ks], acc[u][q],
                                                                0, 0, 0);
      } else {
        const uint32_t off = (uint32_t)s0[u] * (uint32_t)(Cin * 2) + (uint32_t)g * 16u;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8 sf = __builtin_bit_cast(
              bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                          s_rsrc, s0[u] >= 0 ? off + (uint32_t)ks * 64u : kSpOutOfRange, 0, 0));
#pragma unroll
          for (int q = 0; q < NCTW; ++q)
            acc[u][q] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wreg[ks][q], sf, acc[u][q], 0, 0,
                                                                0);
        }
      }
      // activation, bf16 (round to nearest even), 8 bytes per lane and block
      const uint32_t ooff = (uint32_t)row[u] * (uint32_t)(Cout * 2) +
                            (uint32_t)(wave * NCTW) * 32u + (uint32_t)g * 8u;
#pragma unroll
      for (int q = 0; q < NCTW; ++q) {
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float x = acc[u][q][r];
          v[r] = relu ? (x > 0.f ? x : 0.f) : x;
        }
        const sp_bf16x2 h0 = __builtin_convertvector(sp_f32x2{v[0], v[1]}, sp_bf16x2);
        const sp_bf16x2 h1 = __builtin_convertvector(sp_f32x2{v[2], v[3]}, sp_bf16x2);
        const sp_v2u32 w = {__builtin_bit_cast(uint32_t, h0), __builtin_bit_cast(uint32_t, h1)};
        __builtin_amdgcn_raw_buffer_store_b64(
            w, o_rsrc, row[u] < n ? ooff + (uint32_t)q * 32u : kSpOutOfRange, 0, 0);
      }
    }
    if (more) store_rows(buf ^ 1);
    sp_lds_barrier();
    buf ^= 1;
  }
}

template <typename Kern>
hipError_t sp_allow_lds(Kern kern, std::once_flag& once, hipError_t& err) {
  std::call_once(once, [&] {
    err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, kSpLdsLimit);
  });
  return err;
}

// "Big" shapes (a slot's weights at 64 KB or more, or 256 output columns)
// stage the weights in two slices; either launch then fits two workgroups
// per CU.
constexpr bool split_big(int wbytes, int nct) { return wbytes >= 64 * 1024 || nct >= 16; }
constexpr int kSplitWgsPerCu = 2;

// Rows per pair workgroup: about kSplitWgsPerCu workgroups per CU over the
// K - 1 slots, a multiple of 64, within one pass of the table loads and the
// LDS left beside the weights / staging region (`region` bytes).
int split_chunk_rows(int64_t n, int32_t K, int num_cus, int region) {
  const int64_t slots = K > 1 ? K - 1 : 1;
  const int64_t wgs = (int64_t)num_cus * kSplitWgsPerCu;
  int64_t chunks = (wgs + slots - 1) / slots;
  if (chunks < 1) chunks = 1;
  int64_t rc = (n + chunks - 1) / chunks;
  rc = (rc + 63) / 64 * 64;
  const int64_t lds_rows = ((kSpLdsLimit - region - 16) / 6) / 64 * 64;
  if (rc > lds_rows) rc = lds_rows;
  if (rc > kMaxChunkRows) rc = kMaxChunkRows;
  if (rc < 64) rc = 64;
  return (int)rc;
}

// For big shapes one workgroup of either launch fits a CU (the LDS of one
// slot's weights, or the registers of a quarter of 256 columns' fragments).
template <int KS, int NCT>
hipError_t launch_split_k(const SplitArgs& a0, int num_cus, hipStream_t stream) {
  SplitArgs a = a0;
  constexpr int Cin = KS * 32, Cout = NCT * 16;
  constexpr int wbytes = Cin * Cout * 2;
  constexpr bool big = split_big(wbytes, NCT);
  constexpr int WP = big ? 2 : 1;
  if (a.K > 1) {
    a.chunk_rows = split_chunk_rows(a.n_rows, a.K, num_cus, sp_pair_region(Cin, Cout, WP));
    auto kp = conv_pairs_kernel<KS, NCT, WP>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    if (sp_allow_lds(kp, once, err) != hipSuccess) return err;
    const size_t lds = (size_t)sp_pair_region(Cin, Cout, WP) + 6 * (size_t)a.chunk_rows + 16;
    const unsigned chunks = (unsigned)((a.n_rows + a.chunk_rows - 1) / a.chunk_rows);
    hipLaunchKernelGGL(kp, dim3(chunks, (unsigned)(a.K - 1)), dim3(kPairThreads), lds, stream, a);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  // row workgroups: two per CU; for big shapes W[0] is staged in two slices
  // and a batch has two blocks (one at 256 x 256: the fragments of a quarter
  // of W[0] and a batch's accumulators then fill a wavefront's registers)
  constexpr int RB = big ? (KS * NCT >= 128 ? 1 : 2) : kRowBatch;
  const int64_t batches = (a.n_rows + RB * 16 - 1) / (RB * 16);
  int64_t grid = batches;
  const int64_t cap = (int64_t)num_cus * kSplitWgsPerCu;
  if (grid > cap) grid = cap;
  const size_t lds = (size_t)sp_row_region(Cin, Cout, RB, WP);
  if (a.K <= 12) {
    auto kr = conv_rows_kernel<KS, NCT, 3, 2, RB, WP>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    if (sp_allow_lds(kr, once, err) != hipSuccess) return err;
    hipLaunchKernelGGL(kr, dim3((unsigned)grid), dim3(kPairThreads), lds, stream, a);
  } else {
    auto kr = conv_rows_kernel<KS, NCT, 8, 2, RB, WP>;
    static std::once_flag once;
    static hipError_t err = hipSuccess;
    if (sp_allow_lds(kr, once, err) != hipSuccess) return err;
    hipLaunchKernelGGL(kr, dim3((unsigned)grid), dim3(kPairThreads), lds, stream, a);
  }
  return hipGetLastError();
}

bool split_channels_ok(int32_t C) { return C == 64 || C == 128 || C == 256; }

}  // namespace

int64_t conv_split_workspace_bytes(int64_t n_rows, int32_t K, int32_t Cout) {
  return (int64_t)(K > 1 ? K - 1 : 0) * n_rows * Cout * 4;
}

bool conv_split_supported(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout) {
  if (K < 1 || K > 32) return false;
  if (!split_channels_ok(Cin) || !split_channels_ok(Cout)) return false;
  // 32-bit buffer offsets into S, out and the workspace
  if (n_rows * Cin * 2 > 0x7FFF0000LL || n_rows * Cout * 2 > 0x7FFF0000LL) return false;
  return (int64_t)(K > 1 ? K - 1 : 1) * n_rows * Cout * 4 <= 0x7FFF0000LL;
}

hipError_t launch_conv_split(const void* S, const int32_t* table, int64_t n_rows, int32_t K,
                             const void* W, const float* bias, int32_t Cin, int32_t Cout,
                             int32_t relu, void* out, float* workspace, int num_cus,
                             hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  SplitArgs a{};
  a.S = S;
  a.table = table;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.P = workspace;
  a.n_rows = n_rows;
  a.K = K;
  a.relu = relu;
#define SHC_SPLIT_CASE(CI, CO)                                                      \
  if (Cin == CI && Cout == CO) return launch_split_k<CI / 32, CO / 16>(a, num_cus, stream);
  SHC_SPLIT_CASE(64, 64) SHC_SPLIT_CASE(64, 128) SHC_SPLIT_CASE(64, 256)
  SHC_SPLIT_CASE(128, 64) SHC_SPLIT_CASE(128, 128) SHC_SPLIT_CASE(128, 256)
  SHC_SPLIT_CASE(256, 64) SHC_SPLIT_CASE(256, 128) SHC_SPLIT_CASE(256, 256)
#undef SHC_SPLIT_CASE
  return hipErrorInvalidValue;
}

}  // namespace shc
