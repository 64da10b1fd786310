// Mask scores (Eq. 3).  For K masks with aligned outputs O_k [N][C] (bf16,
// stored mask-major as O [K][N][C]):
//
//   F[i][k] = || O_i^T O_k ||_F^2,
//   sim[i][k] = F[i][k] / sqrt(F[i][i] F[k][k]),
//   alpha_out[k] = alpha_in[k] + 1/(K-1) * sum_{i != k} (1 - sim[i][k]),
//
// and the kappa masks of largest alpha_out (ties to the lower index).
//
// Three launches:
//   1. tiles  -- for C in {64, 128, 256}, when little is padded: blocks of
//                256 x 256 of the concatenated outputs' Gram matrix (see
//                gram_block_kernel); otherwise:
//                workgroup (pair i <= k, T x T tile of O_i^T O_k, row split s)
//                accumulates its rows' part of the tile with MFMAs.  Rows go
//                through one LDS stage (padded rows) 128 at a time; the next
//                step's rows are loaded into registers while a step is
//                multiplied, so each workgroup keeps 64 KB (T = 128) in
//                flight.  Exactly the workgroups that fit at once are
//                launched;
//                both operands are read with transposing LDS reads, since the
//                reduction runs over rows: lane (g, l) gets rows 8g .. 8g+7 of
//                channel l.  Four wavefronts, each a (T/2) x (T/2) quarter.
//                The fp32 partial tile goes to the workspace;
//   2. reduce -- per (pair, tile, chunk of entries): the splits summed in a
//                fixed order in fp64, each entry squared, summed -> the
//                chunk's share of F;
//   3. score  -- one workgroup: F per pair, similarities, alpha, ranks.
// Every sum has a fixed order, so the results repeat bit for bit.
#include <algorithm>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kGramThreads = 256;
constexpr int kBlockThreads = 512;
constexpr int kXcds = 8;
constexpr int kCus = 256;
// Rows per step of the tile kernel (both tile edges) and the workgroups of it
// that fit on one CU: at T = 128, 240 registers per lane and 68 KB of LDS
// allow 2; at T = 64, 112 registers and 36 KB allow 4.
constexpr int kRowsPerStep = 128;
__host__ inline int tiles_per_cu(int T) { return T == 128 ? 2 : 4; }
constexpr int kMaxSplits = 512;
constexpr int kScoreThreads = 256;
#define SHC_LDS __attribute__((address_space(3)))
typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));

__host__ __device__ inline int tile_of(int C) { return C % 128 == 0 ? 128 : 64; }

// T: tile edge (64 or 128).  Grid: pairs * tiles * splits workgroups, one
// dimension.  Workgroups are dealt to the 8 XCDs in turn (block b to XCD
// b % 8); the logical index gives each XCD a contiguous run, split-major, so
// the workgroups that read the same rows of a mask share that XCD's L2.
template <int T, int R>
__global__ __launch_bounds__(kGramThreads) void gram_tile_kernel(const __bf16* __restrict__ O,
                                                                 int32_t K, int64_t N, int32_t C,
                                                                 int64_t rows_per_split,
                                                                 int32_t splits,
                                                                 float* __restrict__ part) {
  constexpr int NB = T / 32;                // 16-column blocks per wavefront and side
  constexpr int ROW = T * 2 + 16;           // padded LDS row (bytes)
  constexpr int VPR = T * 2 / 16;           // 16-byte vectors per staged row
  constexpr int LOADS = 2 * R * VPR / kGramThreads;  // per thread per step
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][R * ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int wa = wave >> 1, wb = wave & 1;  // the wave's quarter of the tile
  const int tiles_side = C / T;
  const int tiles = tiles_side * tiles_side;
  const int n_wg = (int)gridDim.x;
  const int xcd = (int)blockIdx.x % kXcds, slot = (int)blockIdx.x / kXcds;
  const int q8 = n_wg / kXcds, r8 = n_wg % kXcds;
  const int logical = (xcd < r8 ? xcd * (q8 + 1) : r8 * (q8 + 1) + (xcd - r8) * q8) + slot;
  const int items = n_wg / splits;
  const int split = logical / items;
  const int pt = logical - split * items;
  const int p = pt / tiles, t = pt - p * tiles;
  const int ta = t / tiles_side, tb = t - ta * tiles_side;
  // pair p -> (i, k), i <= k, row-major over the upper triangle
  int i = 0, rem = p;
  while (rem >= K - i) {
    rem -= K - i;
    ++i;
  }
  const int k = i + rem;
  const int64_t r0 = (int64_t)split * rows_per_split;
  const int64_t r1 = min(r0 + rows_per_split, N);
  const int steps = r1 > r0 ? (int)((r1 - r0 + R - 1) / R) : 0;

  const __bf16* Oa = O + (int64_t)i * N * C + (int64_t)ta * T;
  const __bf16* Ob = O + (int64_t)k * N * C + (int64_t)tb * T;

  auto load = [&](int step, i32x4* v) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int e = tid + u * kGramThreads;  // [operand][row][vector]
      const int op = e / (R * VPR);
      const int rr = (e / VPR) % R;
      const int q = e % VPR;
      const int64_t r = r0 + (int64_t)step * R + rr;
      const __bf16* src = (op == 0 ? Oa : Ob) + (r < r1 ? r : r0) * C + q * 8;
      v[u] = r < r1 ? *reinterpret_cast<const i32x4*>(src) : i32x4{0, 0, 0, 0};
    }
  };
  auto store = [&](const i32x4* v) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int e = tid + u * kGramThreads;
      const int op = e / (R * VPR);
      const int rr = (e / VPR) % R;
      const int q = e % VPR;
      *reinterpret_cast<i32x4*>(&stage[op][rr * ROW + q * 16]) = v[u];
    }
  };
  // rows 8g .. 8g+7 of channel 16 cb + l16 of one staged operand
  auto frag = [&](const unsigned char* base, int cb) -> bf16x8 {
    const unsigned char* p0 = base + (8 * g + (l16 >> 2)) * ROW + cb * 32 + 8 * (l16 & 3);
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0)));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0 + 4 * ROW)));
    return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[NB][NB];
#pragma unroll
  for (int x = 0; x < NB; ++x)
#pragma unroll
    for (int y = 0; y < NB; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  // One LDS stage: the next step's rows are in flight in registers while
  // this step's are multiplied.
  i32x4 v[LOADS];
  if (steps > 0) load(0, v);
  for (int s = 0; s < steps; ++s) {
    store(v);
    __syncthreads();
    if (s + 1 < steps) load(s + 1, v);
#pragma unroll
    for (int sub = 0; sub < R / 32; ++sub) {
      bf16x8 fa[NB], fb[NB];
#pragma unroll
      for (int x = 0; x < NB; ++x) fa[x] = frag(stage[0] + sub * 32 * ROW, wa * NB + x);
#pragma unroll
      for (int y = 0; y < NB; ++y) fb[y] = frag(stage[1] + sub * 32 * ROW, wb * NB + y);
#pragma unroll
      for (int x = 0; x < NB; ++x)
#pragma unroll
        for (int y = 0; y < NB; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[x], fb[y], acc[x][y], 0, 0, 0);
    }
    __syncthreads();
  }
  // partial tile, row-major [T][T]: lane (g, l16) holds rows 4g .. 4g+3 of column l16
  float* out = part + ((int64_t)pt * splits + split) * T * T;
#pragma unroll
  for (int x = 0; x < NB; ++x)
#pragma unroll
    for (int y = 0; y < NB; ++y)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int a = (wa * NB + x) * 16 + 4 * g + rr;
        const int b = (wb * NB + y) * 16 + l16;
        out[a * T + b] = acc[x][y][rr];
      }
}

// Gram blocks of the concatenated outputs M = [O_0 | ... | O_{K-1}] (N rows,
// K C columns, mask-major), for C in {64, 128, 256}, i.e. 256 / C masks per
// 256-column block.  Workgroup (block pair ba <= bb, row split) accumulates
// M[:, 256 ba ..]^T M[:, 256 bb ..] over its rows: twice the flops per loaded
// byte of the T x T pair tiles above.  Four wavefronts, each a 128 x 128
// quarter (64 accumulator blocks); rows go through one padded LDS stage R at
// a time, the next step loaded into registers meanwhile.  Workgroups are
// dealt to the XCDs split-major, as for the pair tiles.
template <int R>
__global__ __launch_bounds__(kBlockThreads) void gram_block_kernel(const __bf16* __restrict__ O, int32_t K, int64_t N, int32_t C,
                       int64_t rows_per_split, int32_t splits, int32_t nb,
                       float* __restrict__ part) {
  constexpr int T = 256;
  constexpr int NA = 8, NBB = 4;              // 16-column blocks per wavefront: A side, B side
  constexpr int ROW = T * 2 + 16;             // padded LDS row (bytes)
  constexpr int VPR = T * 2 / 16;             // 16-byte vectors per staged row
  constexpr int LOADS = 2 * R * VPR / kBlockThreads;
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][R * ROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int wa = wave >> 2, wb = wave & 3;  // the wave's 128 x 64 part of the block
  const int n_wg = (int)gridDim.x;
  const int xcd = (int)blockIdx.x % kXcds, slot = (int)blockIdx.x / kXcds;
  const int q8 = n_wg / kXcds, r8 = n_wg % kXcds;
  const int logical = (xcd < r8 ? xcd * (q8 + 1) : r8 * (q8 + 1) + (xcd - r8) * q8) + slot;
  const int items = n_wg / splits;
  const int split = logical / items;
  const int item = logical - split * items;
  // item -> block pair (ba, bb), ba <= bb, row-major over the upper triangle
  int ba = 0, rem = item;
  while (rem >= nb - ba) {
    rem -= nb - ba;
    ++ba;
  }
  const int bb = ba + rem;
  const int64_t KC = (int64_t)K * C;
  const int64_t r0 = (int64_t)split * rows_per_split;
  const int64_t r1 = min(r0 + rows_per_split, N);
  const int steps = r1 > r0 ? (int)((r1 - r0 + R - 1) / R) : 0;

  // A thread moves one 16-byte column vector q of rows rbase, rbase + RSTEP,
  // ... of both operands; its mask and channel are fixed per operand.
  constexpr int RSTEP = kBlockThreads / VPR;
  constexpr int LPO = LOADS / 2;  // loads per operand and step
  static_assert(RSTEP * LPO == R, "rows per step");
  const int q = tid % VPR, rbase = tid / VPR;
  const int64_t colA = (int64_t)ba * T + q * 8, colB = (int64_t)bb * T + q * 8;
  const bool okA = colA < KC, okB = colB < KC;
  const __bf16* baseA = O + (okA ? (colA / C) * N * C + colA % C : 0);
  const __bf16* baseB = O + (okB ? (colB / C) * N * C + colB % C : 0);
  auto load = [&](int step, i32x4* v) {
#pragma unroll
    for (int u = 0; u < LPO; ++u) {
      const int64_t r = r0 + (int64_t)step * R + rbase + u * RSTEP;
      const bool okr = r < r1;
      v[u] = (okA && okr) ? *reinterpret_cast<const i32x4*>(baseA + r * C) : i32x4{0, 0, 0, 0};
      v[LPO + u] =
          (okB && okr) ? *reinterpret_cast<const i32x4*>(baseB + r * C) : i32x4{0, 0, 0, 0};
    }
  };
  auto store = [&](const i32x4* v) {
#pragma unroll
    for (int u = 0; u < LPO; ++u) {
      const int rr = rbase + u * RSTEP;
      *reinterpret_cast<i32x4*>(&stage[0][rr * ROW + q * 16]) = v[u];
      *reinterpret_cast<i32x4*>(&stage[1][rr * ROW + q * 16]) = v[LPO + u];
    }
  };
  // rows 8g .. 8g+7 of channel 16 cb + l16 of one staged operand
  auto frag = [&](const unsigned char* base, int cb) -> bf16x8 {
    const unsigned char* p0 = base + (8 * g + (l16 >> 2)) * ROW + cb * 32 + 8 * (l16 & 3);
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0)));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0 + 4 * ROW)));
    return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  f32x4 acc[NA][NBB];
#pragma unroll
  for (int x = 0; x < NA; ++x)
#pragma unroll
    for (int y = 0; y < NBB; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};

  i32x4 v[LOADS];
  if (steps > 0) load(0, v);
  for (int st = 0; st < steps; ++st) {
    store(v);
    __syncthreads();
    if (st + 1 < steps) load(st + 1, v);
#pragma unroll
    for (int sub = 0; sub < R / 32; ++sub) {
      bf16x8 fb[NBB];
#pragma unroll
      for (int y = 0; y < NBB; ++y) fb[y] = frag(stage[1] + sub * 32 * ROW, wb * NBB + y);
#pragma unroll
      for (int x = 0; x < NA; ++x) {
        const bf16x8 fa = frag(stage[0] + sub * 32 * ROW, wa * NA + x);
#pragma unroll
        for (int y = 0; y < NBB; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa, fb[y], acc[x][y], 0, 0, 0);
      }
    }
    __syncthreads();
  }
  // partial block, row-major [T][T]: lane (g, l16) holds rows 4g .. 4g+3 of column l16
  float* out = part + ((int64_t)item * splits + split) * T * T;
#pragma unroll
  for (int x = 0; x < NA; ++x)
#pragma unroll
    for (int y = 0; y < NBB; ++y)
#pragma unroll
      for (int rr = 0; rr < 4; ++rr) {
        const int a = (wa * NA + x) * 16 + 4 * g + rr;
        const int b = (wb * NBB + y) * 16 + l16;
        out[a * T + b] = acc[x][y][rr];
      }
}

// Workgroup (sub-block sq of a block pair, chunk of 256 entries): the C x C
// sub-block of masks (i, k), i = ba m + ii, k = bb m + kk (m = 256 / C masks
// per block), i <= k: each entry summed over the splits (fp64, split order),
// squared, and summed -> fq[pair(i, k) * chunks + chunk], the layout the
// score kernel reads.  Sub-blocks with i > k (the transposed half of a
// diagonal block) or past the last mask write nothing.
__global__ __launch_bounds__(256) void gram_block_reduce_kernel(const float* __restrict__ part,
                                                               int splits, int32_t K, int32_t C,
                                                               int32_t nb, int chunks,
                                                               double* __restrict__ fq) {
  __shared__ double red[256];
  const int m = 256 / C;
  const int sq = blockIdx.x;
  const int item = sq / (m * m);
  const int ii = (sq / m) % m, kk = sq % m;
  int ba = 0, rem = item;
  while (rem >= nb - ba) {
    rem -= nb - ba;
    ++ba;
  }
  const int bb = ba + rem;
  const int i = ba * m + ii, k = bb * m + kk;
  if (i >= K || k >= K || i > k) return;
  const float* base = part + (int64_t)item * splits * 65536;
  const int e = blockIdx.y * 256 + threadIdx.x;  // entry of the C x C sub-block
  const int a = ii * C + e / C, b = kk * C + e % C;
  double s = 0.0;
#pragma unroll 8
  for (int q = 0; q < splits; ++q) s += (double)base[(int64_t)q * 65536 + a * 256 + b];
  red[threadIdx.x] = s * s;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    const int p = i * K - i * (i - 1) / 2 + (k - i);
    fq[(int64_t)p * chunks + blockIdx.y] = red[0];
  }
}

// Workgroup (pair-tile pt, chunk j): the entries e = j*256 + tid, + 256*chunks,
// ... of tile pt, each summed over the splits (fp64, split order), squared, and
// summed -> fq[pt * chunks + j].  One entry per thread at a time, so the loads
// of consecutive splits are independent of each other and stay in flight.
__global__ __launch_bounds__(256) void gram_reduce_kernel(const float* __restrict__ part,
                                                          int splits, int TT, int chunks,
                                                          double* __restrict__ fq) {
  __shared__ double red[256];
  const float* base = part + (int64_t)blockIdx.x * splits * TT;
  double acc = 0.0;
  for (int e = blockIdx.y * 256 + threadIdx.x; e < TT; e += 256 * chunks) {
    double s = 0.0;
#pragma unroll 8
    for (int q = 0; q < splits; ++q) s += (double)base[(int64_t)q * TT + e];
    acc += s * s;
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int w = 128; w > 0; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) fq[(int64_t)blockIdx.x * chunks + blockIdx.y] = red[0];
}

__device__ inline int pair_index(int i, int k, int K) {  // i <= k
  return i * K - i * (i - 1) / 2 + (k - i);
}

// One workgroup of kScoreThreads threads.  F of each pair: a wavefront per
// pair sums its parts (lane j: parts j, j + 64, ...; then a fixed butterfly
// over the lanes).  Then thread k < K owns mask k.
__global__ __launch_bounds__(kScoreThreads) void score_kernel(
    const double* __restrict__ fq, int parts, int32_t K, const double* __restrict__ alpha_in,
    double* __restrict__ alpha_out, double* __restrict__ sim, int32_t kappa,
    int32_t* __restrict__ top) {
  __shared__ double F[kMaxScoreMasks * (kMaxScoreMasks + 1) / 2];
  __shared__ double a[kMaxScoreMasks];
  const int P = K * (K + 1) / 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int p = wave; p < P; p += kScoreThreads / 64) {
    double s = 0.0;
    for (int t = lane; t < parts; t += 64) s += fq[(int64_t)p * parts + t];
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) s += __shfl_xor(s, m);
    if (lane == 0) F[p] = s;
  }
  __syncthreads();
  const int k = threadIdx.x;
  if (k < K) {
    const double fkk = F[pair_index(k, k, K)];
    double acc = 0.0;
    for (int i = 0; i < K; ++i) {
      const double fik = F[i <= k ? pair_index(i, k, K) : pair_index(k, i, K)];
      const double fii = F[pair_index(i, i, K)];
      const double den = sqrt(fii * fkk);
      const double sk = den > 0.0 ? fik / den : 1.0;
      if (sim != nullptr) sim[(int64_t)i * K + k] = sk;
      if (i != k) acc += 1.0 - sk;
    }
    const double base = alpha_in != nullptr ? alpha_in[k] : 0.0;
    a[k] = K > 1 ? base + acc / (double)(K - 1) : base;
    alpha_out[k] = a[k];
  }
  __syncthreads();
  if (k < K && top != nullptr) {
    int rank = 0;
    for (int j = 0; j < K; ++j) rank += (a[j] > a[k] || (a[j] == a[k] && j < k)) ? 1 : 0;
    if (rank < kappa) top[rank] = k;
  }
}

}  // namespace

void mask_scores_plan(int32_t K, int64_t N, int32_t C, int* tile, int* tiles, int* splits,
                      int64_t* rows_per_split, int* chunks) {
  const int T = tile_of(C);
  const int side = C / T;
  const int P = K * (K + 1) / 2;
  *tile = T;
  *tiles = side * side;
  const int64_t items = (int64_t)P * side * side;
  // As many row splits as keep every workgroup resident at once (a partial
  // second wave of workgroups would double the time), at least 256 rows each.
  // Each workgroup keeps one step of rows in flight, so the number resident
  // sets the memory parallelism.
  int64_t s = (int64_t)kCus * tiles_per_cu(T) / items;
  const int64_t max_s = std::max<int64_t>(1, (N + 255) / 256);
  s = std::min<int64_t>(std::max<int64_t>(s, 1), std::min<int64_t>(kMaxSplits, max_s));
  *splits = (int)s;
  int64_t rps = (N + s - 1) / s;
  rps = (rps + kRowsPerStep - 1) / kRowsPerStep * kRowsPerStep;
  *rows_per_split = std::max<int64_t>(rps, kRowsPerStep);
  // reduction: about 2048 workgroups, at most one 256-entry chunk each
  int ch = 1;
  while (ch * 256 < T * T && items * ch < 2048) ch *= 2;
  *chunks = ch;
}

namespace {

constexpr int kBlockRows = 64;  // rows per step of the block kernel

// The block path computes nb (nb + 1) / 2 blocks of 256 x 256 where the pairs
// need K (K + 1) / 2 tiles of C x C; with an odd number of masks per block
// row the padding can double the work.  Blocks are taken when they compute
// at most 30% more than the pairs need.
bool use_blocks(int32_t K, int32_t C) {
  if (C != 64 && C != 128 && C != 256) return false;
  const int64_t m = 256 / C, nb = (K + m - 1) / m;
  const int64_t block_area = nb * (nb + 1) / 2 * 65536;
  const int64_t pair_area = (int64_t)K * (K + 1) / 2 * C * C;
  return 10 * block_area <= 13 * pair_area;
}

// Block path: m masks per 256-column block, nb blocks, items = block pairs;
// one workgroup per CU (its LDS stage is 132 KB), so as many row splits as
// fill the CUs once.
struct BlockPlan {
  int m, nb, items, splits, chunks;
  int64_t rps;
};

BlockPlan block_plan(int32_t K, int64_t N, int32_t C) {
  BlockPlan b;
  b.m = 256 / C;
  b.nb = (K + b.m - 1) / b.m;
  b.items = b.nb * (b.nb + 1) / 2;
  int64_t sp = std::max<int64_t>(1, (int64_t)kCus / b.items);
  sp = std::min<int64_t>(sp, std::min<int64_t>(kMaxSplits, (N + kBlockRows - 1) / kBlockRows));
  b.splits = (int)std::max<int64_t>(sp, 1);
  int64_t rps = (N + b.splits - 1) / b.splits;
  b.rps = std::max<int64_t>((rps + kBlockRows - 1) / kBlockRows * kBlockRows, kBlockRows);
  b.chunks = C * C / 256;
  return b;
}

}  // namespace

size_t mask_scores_workspace_bytes(int32_t K, int64_t N, int32_t C) {
  const int64_t P = (int64_t)K * (K + 1) / 2;
  if (use_blocks(K, C)) {
    const BlockPlan b = block_plan(K, N, C);
    const size_t part = (size_t)b.items * b.splits * 65536 * sizeof(float);
    const size_t fq = (size_t)P * b.chunks * sizeof(double);
    return ((part + 255) & ~(size_t)255) + ((fq + 255) & ~(size_t)255);
  }
  int T, tiles, splits, chunks;
  int64_t rps;
  mask_scores_plan(K, N, C, &T, &tiles, &splits, &rps, &chunks);
  const size_t part = (size_t)P * tiles * splits * T * T * sizeof(float);
  const size_t ft = (size_t)P * tiles * chunks * sizeof(double);
  return ((part + 255) & ~(size_t)255) + ((ft + 255) & ~(size_t)255);
}

hipError_t launch_mask_scores(const void* O, int32_t K, int64_t N, int32_t C,
                              const double* alpha_in, double* alpha_out, double* sim,
                              int32_t kappa, int32_t* top, void* ws, hipStream_t stream) {
  const int64_t P = (int64_t)K * (K + 1) / 2;
  float* part = static_cast<float*>(ws);
  if (use_blocks(K, C)) {
    const BlockPlan b = block_plan(K, N, C);
    const size_t part_bytes = (size_t)b.items * b.splits * 65536 * sizeof(float);
    double* fq = reinterpret_cast<double*>(static_cast<unsigned char*>(ws) +
                                           ((part_bytes + 255) & ~(size_t)255));
    hipLaunchKernelGGL((gram_block_kernel<kBlockRows>), dim3((unsigned)(b.items * b.splits)),
                       dim3(kBlockThreads), 0, stream, static_cast<const __bf16*>(O), K, N, C,
                       b.rps, b.splits, b.nb, part);
    hipError_t err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(gram_block_reduce_kernel, dim3((unsigned)(b.items * b.m * b.m),
                                                      (unsigned)b.chunks),
                       dim3(256), 0, stream, part, b.splits, K, C, b.nb, b.chunks, fq);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    hipLaunchKernelGGL(score_kernel, dim3(1), dim3(kScoreThreads), 0, stream, fq, b.chunks, K,
                       alpha_in, alpha_out, sim, kappa, top);
    return hipGetLastError();
  }
  int T, tiles, splits, chunks;
  int64_t rps;
  mask_scores_plan(K, N, C, &T, &tiles, &splits, &rps, &chunks);
  const size_t part_bytes = (size_t)P * tiles * splits * T * T * sizeof(float);
  double* ft = reinterpret_cast<double*>(static_cast<unsigned char*>(ws) +
                                         ((part_bytes + 255) & ~(size_t)255));
  const dim3 grid((unsigned)(P * tiles * splits));
  if (T == 128)
    hipLaunchKernelGGL((gram_tile_kernel<128, kRowsPerStep>), grid, dim3(kGramThreads), 0, stream,
                       static_cast<const __bf16*>(O), K, N, C, rps, splits, part);
  else
    hipLaunchKernelGGL((gram_tile_kernel<64, kRowsPerStep>), grid, dim3(kGramThreads), 0, stream,
                       static_cast<const __bf16*>(O), K, N, C, rps, splits, part);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(gram_reduce_kernel, dim3((unsigned)(P * tiles), (unsigned)chunks), dim3(256),
                     0, stream, part, splits, T * T, chunks, ft);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(score_kernel, dim3(1), dim3(kScoreThreads), 0, stream, ft, tiles * chunks, K,
                     alpha_in, alpha_out, sim, kappa, top);
  return hipGetLastError();
}

}  // namespace shc
