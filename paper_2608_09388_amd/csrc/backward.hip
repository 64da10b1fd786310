// Backward of the sparse linear layer (Eq. 6) and the sparse neighbourhood
// convolution (Eqs. 4-5), with the ReLU of Eq. 10.  The gradients are those
// of the dense operator on x (.) m restricted to the active rows:
//
//   dZ = dY (.) [Y > 0]                       (Y: the layer's stored output)
//   db[o]       = sum_i dZ[i][o]
//   dW[j][c][o] = sum_{i : r_ij >= 0} S[r_ij][c] dZ[i][o]
//   dS[r][c]    = sum_{(i, j) : r_ij = r} sum_o dZ[i][o] W[j][c][o]
//
// with r_ij the row that slot j of row i reads (the neighbour-row table;
// r_i0 = i and K = 1 for the linear layer).
//
// Kernels:
//   * linear_bwd_fused -- the bf16 linear layer of 64 or 128 channels in one
//     pass over the rows (dZ in registers, dS, partial dW and column sums);
//   * relu_bwd     -- dZ, and per-split column sums of dZ (db, fixed order);
//   * transposed neighbour lists, once per mesh: for vertex u and slot j, the
//     vertices v whose slot j points at u, ascending.  The c-th of them is
//     "virtual slot" (j, c); a mesh has Kt = sum_j max_u |list(u, j)| of them;
//   * transposed table, once per active set: for active row r and virtual
//     slot s = (j, c), the active row that sends to r through it (or -1),
//     plus a 64-bit mask of the virtual slots present in the row;
//   * dgrad (dS)   -- the transposed table makes dS a gathered contraction
//     like the forward one: rows of dZ gathered per virtual slot, times
//     W[j]^T.  A B fragment of W[j]^T (8 consecutive reduction entries o of
//     one output column c) is 16 contiguous bytes of W[j][c][.], so the
//     weights go to LDS in fragment order with plain copies;
//   * wgrad (dW)   -- per slot, the Gram-type contraction S[r_ij]^T dZ[i] over
//     the rows i where slot j is present.  Those rows come from a compaction
//     of the [K][N'] presence mask (slot-major lists, ascending i); each list
//     is cut into chunks of a fixed number of rows, a workgroup multiplies one
//     chunk into a fp32 partial tile, and the partials of a slot are summed in
//     chunk order in fp64.
// Every sum has a fixed order, so results repeat bit for bit.
#include <algorithm>
#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kThreads = 256;
#define SHC_LDS __attribute__((address_space(3)))
typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef uint32_t v4u32 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
constexpr int kBufferWord3 = 0x00020000;
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kMaxSlotsBwd = 32;
constexpr int kWgradRows = 128;      // rows per step of the wgrad tile kernel
// dynamic LDS of the dgrad kernel: 160 KB less room for its static arrays
constexpr int kDgradLds = 159 * 1024;
constexpr int kDgradThreads = 512;
constexpr int kDgradMaxRows = 1536;  // rows per workgroup (sorted in LDS)
constexpr int kWBatch = 8;           // weight vectors per thread in flight while staging

// ---------------------------------------------------------------------------
// dZ and the column sums of db
// ---------------------------------------------------------------------------

// Workgroup s takes rows [s * rps, (s + 1) * rps).  A thread owns one 16-byte
// vector column q of rows y, y + ty, ...; its sums, then the ty row groups in
// order, give colpart[s][c].  With act == 0, dZ = dY and nothing is written.
template <bool BF16>
__global__ __launch_bounds__(kThreads) void relu_bwd_kernel(const i32x4* __restrict__ dY,
                                                            const i32x4* __restrict__ Y,
                                                            int64_t n, int32_t C, int act,
                                                            int64_t rps, i32x4* __restrict__ dZ,
                                                            float* __restrict__ colpart) {
  constexpr int PER = BF16 ? 8 : 4;
  __shared__ float red[kThreads * 8];
  const int vpr = C / PER;
  const int ty = kThreads / vpr;
  const int q = threadIdx.x % vpr, y = threadIdx.x / vpr;
  const int64_t r0 = (int64_t)blockIdx.x * rps;
  const int64_t r1 = min(r0 + rps, n);
  float s[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) s[e] = 0.f;
  if (y < ty) {
    for (int64_t r = r0 + y; r < r1; r += ty) {
      const int64_t idx = r * vpr + q;
      i32x4 g = dY[idx];
      if (act) {
        const i32x4 yv = Y[idx];
        if (BF16) {
#pragma unroll
          for (int w = 0; w < 4; ++w) {
            const uint32_t gw = (uint32_t)g[w], yw = (uint32_t)yv[w];
            const uint32_t lo = bf16_bits_to_f32(yw & 0xFFFFu) > 0.f ? (gw & 0xFFFFu) : 0u;
            const uint32_t hi = bf16_bits_to_f32(yw >> 16) > 0.f ? (gw & 0xFFFF0000u) : 0u;
            g[w] = (int)(lo | hi);
          }
        } else {
#pragma unroll
          for (int w = 0; w < 4; ++w) g[w] = __int_as_float(yv[w]) > 0.f ? g[w] : 0;
        }
        dZ[idx] = g;
      }
      if (BF16) {
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          s[2 * w] += bf16_bits_to_f32((uint32_t)g[w] & 0xFFFFu);
          s[2 * w + 1] += bf16_bits_to_f32((uint32_t)g[w] >> 16);
        }
      } else {
#pragma unroll
        for (int w = 0; w < 4; ++w) s[w] += __int_as_float(g[w]);
      }
    }
  }
#pragma unroll
  for (int e = 0; e < PER; ++e) red[threadIdx.x * 8 + e] = s[e];
  __syncthreads();
  for (int c = threadIdx.x; c < C; c += kThreads) {
    const int qq = c / PER, e = c % PER;
    float t = 0.f;
    for (int yy = 0; yy < ty; ++yy) t += red[(yy * vpr + qq) * 8 + e];
    colpart[(int64_t)blockIdx.x * C + c] = t;
  }
}

// db[c]: workgroup of 8 columns x 32 split groups; group y sums splits y,
// y + 32, ... in fp64, then the 32 group sums are added in order; one rounding.
__global__ __launch_bounds__(kThreads) void colsum_kernel(const float* __restrict__ colpart,
                                                          int splits, int32_t C,
                                                          float* __restrict__ db) {
  __shared__ double red[32][8];
  const int cx = threadIdx.x & 7, y = threadIdx.x >> 3;
  const int c = blockIdx.x * 8 + cx;
  double t = 0.0;
  if (c < C) {
#pragma unroll 4
    for (int s = y; s < splits; s += 32) t += (double)colpart[(int64_t)s * C + c];
  }
  red[y][cx] = t;
  __syncthreads();
  if (y == 0 && c < C) {
    double u = 0.0;
    for (int yy = 0; yy < 32; ++yy) u += red[yy][cx];
    db[c] = (float)u;
  }
}

// ---------------------------------------------------------------------------
// transposed neighbour lists (once per mesh)
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kThreads) void fill_i32_kernel(int32_t* __restrict__ p, int64_t n,
                                                            int32_t v) {
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads)
    p[i] = v;
}

// cnt[u * K + j] = number of v with nbr[v][j] = u
__global__ __launch_bounds__(kThreads) void tv_count_kernel(const int32_t* __restrict__ nbr,
                                                            int32_t V, int32_t K,
                                                            int32_t* __restrict__ cnt) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= (int64_t)V * K) return;
  const int j = (int)(e % K);
  const int32_t u = nbr[e];
  if (u >= 0 && u < V) atomicAdd(&cnt[(int64_t)u * K + j], 1);
}

// One workgroup: m_j = max_u cnt[u][j]; off[j] = sum_{j' < j} m_j'; off[K] = Kt;
// slot_of[s] = j for the virtual slots s of slot j.
__global__ __launch_bounds__(kThreads) void tv_layout_kernel(const int32_t* __restrict__ cnt,
                                                             int32_t V, int32_t K,
                                                             int32_t* __restrict__ off,
                                                             int32_t* __restrict__ slot_of,
                                                             int32_t max_kt) {
  __shared__ int32_t mx[kThreads];
  __shared__ int32_t mj[kMaxSlotsBwd];
  for (int j = 0; j < K; ++j) {
    int32_t m = 0;
    for (int32_t u = threadIdx.x; u < V; u += kThreads) m = max(m, cnt[(int64_t)u * K + j]);
    mx[threadIdx.x] = m;
    __syncthreads();
    for (int w = kThreads / 2; w > 0; w >>= 1) {
      if (threadIdx.x < w) mx[threadIdx.x] = max(mx[threadIdx.x], mx[threadIdx.x + w]);
      __syncthreads();
    }
    if (threadIdx.x == 0) mj[j] = mx[0];
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int32_t o = 0;
    for (int j = 0; j < K; ++j) {
      off[j] = o;
      for (int c = 0; c < mj[j]; ++c)
        if (o + c < max_kt) slot_of[o + c] = j;
      o += mj[j];
    }
    off[K] = o;
  }
}

// tv[u * Kt + off[j] + c] = v for the c-th (arrival order) v with nbr[v][j] = u
__global__ __launch_bounds__(kThreads) void tv_fill_kernel(const int32_t* __restrict__ nbr,
                                                           int32_t V, int32_t K,
                                                           const int32_t* __restrict__ off,
                                                           int32_t* __restrict__ cur,
                                                           int32_t* __restrict__ tv,
                                                           int32_t max_kt) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= (int64_t)V * K) return;
  const int32_t Kt = off[K];
  if (Kt > max_kt) return;  // does not fit: the caller reports it
  const int j = (int)(e % K);
  const int32_t v = (int32_t)(e / K);
  const int32_t u = nbr[e];
  if (u < 0 || u >= V) return;
  const int c = atomicAdd(&cur[(int64_t)u * K + j], 1);
  tv[(int64_t)u * Kt + off[j] + c] = v;
}

// sort each (u, j) run ascending, so the order does not depend on arrival
__global__ __launch_bounds__(kThreads) void tv_sort_kernel(const int32_t* __restrict__ cnt,
                                                           int32_t V, int32_t K,
                                                           const int32_t* __restrict__ off,
                                                           int32_t* __restrict__ tv,
                                                           int32_t max_kt) {
  const int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (e >= (int64_t)V * K) return;
  const int32_t Kt = off[K];
  if (Kt > max_kt) return;
  const int j = (int)(e % K);
  const int64_t u = e / K;
  const int m = cnt[e];
  int32_t* p = tv + u * Kt + off[j];
  for (int a = 1; a < m; ++a) {
    const int32_t x = p[a];
    int b = a - 1;
    while (b >= 0 && p[b] > x) {
      p[b + 1] = p[b];
      --b;
    }
    p[b + 1] = x;
  }
}

// ---------------------------------------------------------------------------
// transposed table of an active set
// ---------------------------------------------------------------------------

// table_t[s * n + i] = inv[b_i * V + tv[v_i * Kt + s]] or -1; row_slots[i] has
// bit s set when that entry is a row.  Four lanes per row, lane q taking the
// virtual slots 16 q .. 16 q + 15 (both load rounds of all four in flight at
// once); the row's mask is or-ed over the four lanes by shuffles.
__global__ __launch_bounds__(kThreads) void tt_kernel(const int2* __restrict__ coords,
                                                      const int32_t* __restrict__ inv, int64_t n,
                                                      int32_t B, int32_t V,
                                                      const int32_t* __restrict__ tv, int32_t Kt,
                                                      int32_t* __restrict__ table_t,
                                                      uint64_t* __restrict__ row_slots) {
  const int64_t gid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t i = gid >> 2;
  const int q = (int)(gid & 3);
  const bool in = i < n;
  const int2 c = coords[in ? i : 0];
  const bool ok = in && c.x >= 0 && c.x < B && c.y >= 0 && c.y < V;
  const int32_t* trow = tv + (int64_t)(ok ? c.y : 0) * Kt;
  const int32_t* irow = inv + (int64_t)(ok ? c.x : 0) * V;
  const int s0 = q * 16;
  int32_t v[16], r[16];
#pragma unroll
  for (int u = 0; u < 16; ++u) v[u] = s0 + u < Kt ? trow[s0 + u] : -1;
#pragma unroll
  for (int u = 0; u < 16; ++u) {
    const bool live = ok && v[u] >= 0 && v[u] < V;
    r[u] = irow[live ? v[u] : 0];
    r[u] = (live && r[u] >= 0 && (int64_t)r[u] < n) ? r[u] : -1;
  }
  uint64_t bits = 0;
#pragma unroll
  for (int u = 0; u < 16; ++u)
    if (in && s0 + u < Kt) {
      table_t[(int64_t)(s0 + u) * n + i] = r[u];
      if (r[u] >= 0) bits |= 1ull << (s0 + u);
    }
  // or over the row's four lanes (lanes 4k .. 4k + 3 of the wavefront)
#pragma unroll
  for (int d = 1; d < 4; d <<= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)bits, d, 64);
    const uint32_t hi = __shfl_xor((uint32_t)(bits >> 32), d, 64);
    bits |= ((uint64_t)hi << 32) | lo;
  }
  if (in && q == 0) row_slots[i] = bits;
}

// ---------------------------------------------------------------------------
// wgrad: presence mask, chunk schedule, partial tiles, reduction
// ---------------------------------------------------------------------------

__global__ __launch_bounds__(kThreads) void presence_kernel(const int32_t* __restrict__ table,
                                                            int64_t total,
                                                            uint8_t* __restrict__ m) {
  for (int64_t e = (int64_t)blockIdx.x * kThreads + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * kThreads)
    m[e] = table[e] >= 0 ? 1 : 0;
}

// chunks of L rows of slot j's list: the first one's index and the count
__device__ inline void slot_chunks(const int32_t* __restrict__ row_ptr, int j, int32_t L,
                                   int* first, int* count) {
  int c = 0;
  for (int q = 0; q < j; ++q) c += (row_ptr[q + 1] - row_ptr[q] + L - 1) / L;
  *first = c;
  *count = (row_ptr[j + 1] - row_ptr[j] + L - 1) / L;
}

// Partial tile of dW[j] over one chunk of slot j's rows.  Workgroup
// (chunk w, tile t); chunks past the last exit.  Pair t of the list is
// (slot j, row i) = pairs[t]; the A row is S[table[j * n + i]], the B row
// dZ[i].  Without a list (linear layer): one slot, row t itself on both sides.
// Layout and MFMA scheme as the Gram tiles of the mask scores: R rows through
// one padded LDS stage, both operands read with transposing reads, four
// wavefronts each a (T/2) x (T/2) quarter.
template <int T, int R>
__global__ __launch_bounds__(kThreads) void wgrad_tile_kernel(
    const __bf16* __restrict__ S, const __bf16* __restrict__ dZ, const int32_t* __restrict__ table,
    const int2* __restrict__ pairs, const int32_t* __restrict__ row_ptr, int32_t K, int64_t n,
    int32_t L, int32_t Cin, int32_t Cout, float* __restrict__ part) {
  constexpr int NB = T / 32;
  constexpr int ROW = T * 2 + 16;
  constexpr int VPR = T * 2 / 16;
  constexpr int LOADS = 2 * R * VPR / kThreads;
  constexpr int kMaxL = 512;
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][R * ROW];
  __shared__ int32_t ia[kMaxL], ib[kMaxL];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int wa = wave >> 1, wb = wave & 1;
  const int tA = (Cin + T - 1) / T, tB = (Cout + T - 1) / T;
  const int tiles = tA * tB;
  const int w = blockIdx.x / tiles, t = blockIdx.x - w * tiles;
  const int ta = t / tB, tb = t - ta * tB;
  int j = 0;
  int64_t t0, t1;
  if (pairs != nullptr) {
    // chunk w: slot j and the chunk's place in slot j's list
    int c = 0, wc = -1;
    for (j = 0; j < K; ++j) {
      const int nch = (row_ptr[j + 1] - row_ptr[j] + L - 1) / L;
      if (w < c + nch) {
        wc = w - c;
        break;
      }
      c += nch;
    }
    if (wc < 0) return;  // past the last chunk
    const int64_t base = row_ptr[j] + (int64_t)wc * L;
    t0 = base;
    t1 = min(base + L, (int64_t)row_ptr[j + 1]);
  } else {
    t0 = (int64_t)w * L;
    if (t0 >= n) return;
    t1 = min(t0 + L, n);
  }
  const int rows = (int)(t1 - t0);
  // the chunk's row indices, once
  for (int q = tid; q < rows; q += kThreads) {
    if (pairs != nullptr) {
      const int2 p = pairs[t0 + q];
      const int32_t i = p.y;
      const int32_t a = table[(int64_t)j * n + i];
      ia[q] = a;
      ib[q] = i;
    } else {
      ia[q] = (int32_t)(t0 + q);
      ib[q] = (int32_t)(t0 + q);
    }
  }
  __syncthreads();
  const int steps = (rows + R - 1) / R;

  auto load = [&](int step, i32x4* v) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int e = tid + u * kThreads;
      const int op = e / (R * VPR);
      const int rr = (e / VPR) % R;
      const int q = e % VPR;
      const int local = step * R + rr;
      const int col = (op == 0 ? ta : tb) * T + q * 8;
      const int C = op == 0 ? Cin : Cout;
      v[u] = i32x4{0, 0, 0, 0};
      if (local < rows && col < C) {
        const int32_t row = op == 0 ? ia[local] : ib[local];
        if (row >= 0)
          v[u] = *reinterpret_cast<const i32x4*>((op == 0 ? S : dZ) + (int64_t)row * C + col);
      }
    }
  };
  auto store = [&](const i32x4* v) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int e = tid + u * kThreads;
      const int op = e / (R * VPR);
      const int rr = (e / VPR) % R;
      const int q = e % VPR;
      *reinterpret_cast<i32x4*>(&stage[op][rr * ROW + q * 16]) = v[u];
    }
  };
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
  float* out = part + ((int64_t)w * tiles + t) * T * T;
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

// fp32 version of the partial tiles: T = 64, R = 32 rows per step, one LDS
// stage (rows padded by 64 bytes, so the four row groups of a read sit in
// different banks), the next step in registers.  MFMA 16x16x4 (fp32): lane
// (g, i) gives row g of the k-step at channel i on both sides; the output
// layout is that of the bf16 tiles.
template <int T, int R>
__global__ __launch_bounds__(kThreads) void wgrad_tile_f32_kernel(
    const float* __restrict__ S, const float* __restrict__ dZ, const int32_t* __restrict__ table,
    const int2* __restrict__ pairs, const int32_t* __restrict__ row_ptr, int32_t K, int64_t n,
    int32_t L, int32_t Cin, int32_t Cout, float* __restrict__ part) {
  constexpr int NB = T / 32;
  constexpr int ROW = T * 4 + 64;  // bytes
  constexpr int VPR = T * 4 / 16;
  constexpr int LOADS = 2 * R * VPR / kThreads;
  constexpr int kMaxL = 512;
  __shared__ __attribute__((aligned(16))) unsigned char stage[2][R * ROW];
  __shared__ int32_t ia[kMaxL], ib[kMaxL];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int wa = wave >> 1, wb = wave & 1;
  const int tA = (Cin + T - 1) / T, tB = (Cout + T - 1) / T;
  const int tiles = tA * tB;
  const int w = blockIdx.x / tiles, t = blockIdx.x - w * tiles;
  const int ta = t / tB, tb = t - ta * tB;
  int j = 0;
  int64_t t0, t1;
  if (pairs != nullptr) {
    int c = 0, wc = -1;
    for (j = 0; j < K; ++j) {
      const int nch = (row_ptr[j + 1] - row_ptr[j] + L - 1) / L;
      if (w < c + nch) {
        wc = w - c;
        break;
      }
      c += nch;
    }
    if (wc < 0) return;  // past the last chunk
    const int64_t base = row_ptr[j] + (int64_t)wc * L;
    t0 = base;
    t1 = min(base + L, (int64_t)row_ptr[j + 1]);
  } else {
    t0 = (int64_t)w * L;
    if (t0 >= n) return;
    t1 = min(t0 + L, n);
  }
  const int rows = (int)(t1 - t0);
  for (int q = tid; q < rows; q += kThreads) {
    if (pairs != nullptr) {
      const int2 pq = pairs[t0 + q];
      ia[q] = table[(int64_t)j * n + pq.y];
      ib[q] = pq.y;
    } else {
      ia[q] = (int32_t)(t0 + q);
      ib[q] = (int32_t)(t0 + q);
    }
  }
  __syncthreads();
  const int steps = (rows + R - 1) / R;
  auto load = [&](int step, i32x4* v) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int e = tid + u * kThreads;
      const int op = e / (R * VPR);
      const int rr = (e / VPR) % R;
      const int q = e % VPR;
      const int local = step * R + rr;
      const int col = (op == 0 ? ta : tb) * T + q * 4;
      const int C = op == 0 ? Cin : Cout;
      v[u] = i32x4{0, 0, 0, 0};
      if (local < rows && col < C) {
        const int32_t row = op == 0 ? ia[local] : ib[local];
        if (row >= 0)
          v[u] = *reinterpret_cast<const i32x4*>((op == 0 ? S : dZ) + (int64_t)row * C + col);
      }
    }
  };
  auto store = [&](const i32x4* v) {
#pragma unroll
    for (int u = 0; u < LOADS; ++u) {
      const int e = tid + u * kThreads;
      const int op = e / (R * VPR);
      const int rr = (e / VPR) % R;
      const int q = e % VPR;
      *reinterpret_cast<i32x4*>(&stage[op][rr * ROW + q * 16]) = v[u];
    }
  };
  f32x4 acc[NB][NB];
#pragma unroll
  for (int x = 0; x < NB; ++x)
#pragma unroll
    for (int y = 0; y < NB; ++y) acc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
  i32x4 v[LOADS];
  if (steps > 0) load(0, v);
  for (int st = 0; st < steps; ++st) {
    store(v);
    __syncthreads();
    if (st + 1 < steps) load(st + 1, v);
#pragma unroll
    for (int k0 = 0; k0 < R; k0 += 4) {
      float fa[NB], fb[NB];
#pragma unroll
      for (int x = 0; x < NB; ++x)
        fa[x] = *reinterpret_cast<const float*>(
            &stage[0][(k0 + g) * ROW + ((wa * NB + x) * 16 + l16) * 4]);
#pragma unroll
      for (int y = 0; y < NB; ++y)
        fb[y] = *reinterpret_cast<const float*>(
            &stage[1][(k0 + g) * ROW + ((wb * NB + y) * 16 + l16) * 4]);
#pragma unroll
      for (int x = 0; x < NB; ++x)
#pragma unroll
        for (int y = 0; y < NB; ++y)
          acc[x][y] = __builtin_amdgcn_mfma_f32_16x16x4f32(fa[x], fb[y], acc[x][y], 0, 0, 0);
    }
    __syncthreads();
  }
  float* out = part + ((int64_t)w * tiles + t) * T * T;
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

// dW[j][c][o]: sum of the partial tiles of slot j's chunks in fp64.
// Workgroup (slot j and tile, 32 consecutive entries) of G chunk groups:
// group y sums chunks y, y + G, ... of the slot in order, then the G group
// sums are added in order.  A slot without chunks gets 0.  G = 32 for the
// linear layer (one slot with all the chunks), 8 for a conv (whose sparse
// slots have few chunks each).  With colpart, the workgroups of one more x
// index reduce the bias gradient in colsum_kernel's order (32 groups: group y
// sums splits y, y + 32, ..., whatever G is).
template <int T, int G>
__global__ __launch_bounds__(32 * G) void wgrad_reduce_kernel(
    const float* __restrict__ part, const int32_t* __restrict__ row_ptr, int32_t L, int32_t Cin,
    int32_t Cout, int single, int32_t n_chunks, float* __restrict__ dW,
    const float* __restrict__ colpart, int32_t splits, float* __restrict__ db) {
  __shared__ double red[32][33];
  static_assert(G == 8 || G == 32, "chunk groups");
  const int tA = (Cin + T - 1) / T, tB = (Cout + T - 1) / T;
  const int tiles = tA * tB;
  const int ex = threadIdx.x & 31, y = threadIdx.x >> 5;
  const int e = blockIdx.y * 32 + ex;
  // the last x index is the bias gradient's when colpart is given
  if (colpart != nullptr && (int)blockIdx.x == (int)gridDim.x - 1) {
    // 32 split groups over the G * 32 threads (G = 8: four groups per thread)
    for (int yg = y; yg < 32; yg += G) {
      double t = 0.0;
      if (e < Cout) {
#pragma unroll 4
        for (int q = yg; q < splits; q += 32) t += (double)colpart[(int64_t)q * Cout + e];
      }
      red[yg][ex] = t;
    }
    __syncthreads();
    if (y == 0 && e < Cout) {
      double u = 0.0;
      for (int yy = 0; yy < 32; ++yy) u += red[yy][ex];
      db[e] = (float)u;
    }
    return;
  }
  const int j = blockIdx.x / tiles, t = blockIdx.x - j * tiles;
  const int ta = t / tB, tb = t - ta * tB;
  int c0 = 0, c1 = n_chunks;
  if (!single) {
    int cnt;
    slot_chunks(row_ptr, j, L, &c0, &cnt);
    c1 = c0 + cnt;
  }
  // NU chunks' loads in flight at once (clamped addresses, past-the-end
  // values dropped), then added in chunk order; NU covers about a thread's
  // share (the linear layer's one slot has all the chunks)
  constexpr int NU = G >= 32 ? 8 : 4;
  double s = 0.0;
  const int64_t stride = (int64_t)tiles * T * T;
  const float* pe = part + (int64_t)t * T * T + e;
  for (int q0 = c0 + y; q0 < c1; q0 += NU * G) {
    float v[NU];
#pragma unroll
    for (int u = 0; u < NU; ++u) {
      const int q = q0 + u * G;
      v[u] = pe[(int64_t)(q < c1 ? q : q0) * stride];
    }
#pragma unroll
    for (int u = 0; u < NU; ++u)
      if (q0 + u * G < c1) s += (double)v[u];
  }
  red[y][ex] = s;
  __syncthreads();
  if (y == 0) {
    double u = 0.0;
    for (int yy = 0; yy < G; ++yy) u += red[yy][ex];
    const int a = e / T, b = e - a * T;
    const int c = ta * T + a, o = tb * T + b;
    if (c < Cin && o < Cout) dW[((int64_t)j * Cin + c) * Cout + o] = (float)u;
  }
}

// ---------------------------------------------------------------------------
// dgrad: dS through the transposed table
// ---------------------------------------------------------------------------

// Grid: (row groups of R rows) x (column slices of WS input channels);
// kDgradThreads threads.  Workgroup:
//   * the fragments of W[j]^T for every slot j, k-step and 16-column block of
//     its slice go to LDS once (frag f = (j * KS + ks) * NCB + cb, one 1 KB
//     run of 64 lanes x 16 bytes);
//   * with a transposed table, its rows are bucketed (LDS histogram and
//     cursors) by their first sparse virtual slot -- one present in fewer
//     than half of the rows -- so 16-row blocks hold rows that share it;
//     each block's slot mask is the or of its rows' masks;
//   * each wavefront walks its blocks b = wave, wave + 8, ...; a block's
//     jobs are its virtual slots in ascending order (one empty job when it
//     has none).  A job loads the rows' sources through table_t, their dZ
//     rows as A fragments (raw buffer loads, an absent row reading zeros),
//     and runs NCB x KS MFMAs against W[slot_of[s]]^T.  Jobs go through a
//     ring of register sets in two stages (source rows, then data); after a
//     block's last job its 16 rows are rounded and stored, through the
//     wavefront's LDS scratch, at their original positions.
// Every row is accumulated over its virtual slots in ascending order whatever
// block it lands in (absent slots add exact zeros), so the result does not
// depend on the sort.  Without a transposed table (linear layer) every row is
// its own source through one slot, unsorted.
template <int WS, int KSM, bool TBL, bool BF16>
__global__ __launch_bounds__(kDgradThreads) void dgrad_kernel(
    const unsigned char* __restrict__ dZ, const unsigned char* __restrict__ W,
    const int32_t* __restrict__ table_t, const uint64_t* __restrict__ row_slots,
    const int32_t* __restrict__ slot_of, int64_t n, int32_t K, int32_t Cin, int32_t Cout,
    int32_t R, unsigned char* __restrict__ dS) {
  constexpr int E = BF16 ? 2 : 4;          // bytes per element
  constexpr int KW = BF16 ? 32 : 16;       // reduction entries per k-step (64 bytes)
  constexpr int NCB = WS / 16;
  constexpr int DA = KSM <= 4 ? 4 : (KSM <= 8 ? 2 : 1);  // jobs with data loads in flight
  constexpr int D = 2 * DA;              // ring: as many again with only the source loaded
  constexpr int kWaves = kDgradThreads / 64;
  constexpr int RPT = kDgradMaxRows / kDgradThreads;  // rows per thread in the sort
  constexpr int NBK = kMaxVirtualSlots + 1;            // sort buckets
  constexpr int WROW = WS * E + 16;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int KS = (Cout + KW - 1) / KW;
  unsigned char* wl = smem;                                     // [K][KS][NCB][64][16]
  unsigned char* scratch = smem + (size_t)K * KS * NCB * 1024;  // [waves][16][WROW]
  uint64_t* blkmask = reinterpret_cast<uint64_t*>(scratch + kWaves * 16 * WROW);  // [R / 16]
  int32_t* perm = reinterpret_cast<int32_t*>(blkmask + kDgradMaxRows / 16);         // [R]
  int32_t* hist = perm + kDgradMaxRows;                       // [NBK]: counts, then cursors
  __shared__ int32_t slot_lds[kMaxVirtualSlots];
  __shared__ int32_t scnt[kMaxVirtualSlots];
  __shared__ uint64_t dense_lds;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  const int nrows = (int)min((int64_t)R, n - row0);
  const int n0 = blockIdx.y * WS;

  // sort keys' inputs go out with the weights
  uint64_t mrow[RPT];
  if (TBL) {
#pragma unroll
    for (int rr = 0; rr < RPT; ++rr) {
      const int t = tid + rr * kDgradThreads;
      mrow[rr] = t < nrows ? row_slots[row0 + t] : 0ull;
    }
    if (tid < kMaxVirtualSlots) {
      slot_lds[tid] = slot_of[tid];
      scnt[tid] = 0;
    }
    for (int q = tid; q < NBK; q += kDgradThreads) hist[q] = 0;
    for (int b = tid; b < kDgradMaxRows / 16; b += kDgradThreads) blkmask[b] = 0ull;
  }
  // weights: lane (g, l16) of fragment (j, ks, cb) holds the 16 bytes
  // W[j][n0 + 16 cb + l16][KW ks + (KW / 4) g ...] (8 bf16 or 4 fp32 entries);
  // kWBatch vectors per thread in flight at a time
  const int nfrag = K * KS * NCB * 64;
  for (int f0 = 0; f0 < nfrag; f0 += kWBatch * kDgradThreads) {
    i32x4 v[kWBatch];
#pragma unroll
    for (int u = 0; u < kWBatch; ++u) {
      const int f = f0 + u * kDgradThreads + tid;
      const int ln = f & 63;
      const int fr = f >> 6;
      const int cb = fr % NCB;
      const int ks = (fr / NCB) % KS;
      const int j = fr / (NCB * KS);
      const int c = n0 + cb * 16 + (ln & 15);
      const int o = ks * KW + (KW / 4) * (ln >> 4);
      const bool ok = f < nfrag && c < Cin && o < Cout;
      v[u] = *reinterpret_cast<const i32x4*>(W + (ok ? (((int64_t)j * Cin + c) * Cout + o) * E : 0));
      if (!ok) v[u] = i32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int u = 0; u < kWBatch; ++u) {
      const int f = f0 + u * kDgradThreads + tid;
      if (f < nfrag) *reinterpret_cast<i32x4*>(wl + (size_t)f * 16) = v[u];
    }
  }
  __syncthreads();

  if (TBL) {
    // rows per virtual slot (only the slots some row of the wavefront has)
    uint64_t wor = 0;
#pragma unroll
    for (int rr = 0; rr < RPT; ++rr) wor |= mrow[rr];
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t lo = __shfl_xor((uint32_t)wor, d, 64);
      const uint32_t hi = __shfl_xor((uint32_t)(wor >> 32), d, 64);
      wor |= ((uint64_t)hi << 32) | lo;
    }
    wor = ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(wor >> 32)) << 32) |
          (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)wor);
    for (uint64_t bits = wor; bits != 0; bits &= bits - 1) {
      const int sl = __builtin_ctzll(bits);
      int c = 0;
#pragma unroll
      for (int rr = 0; rr < RPT; ++rr) c += __popcll(__ballot((mrow[rr] >> sl) & 1ull));
      if (lane == 0) atomicAdd(&scnt[sl], c);
    }
    __syncthreads();
    if (wave == 0) {
      const uint64_t d = __ballot(lane < kMaxVirtualSlots && 2 * scnt[lane] >= nrows);
      if (lane == 0) dense_lds = d;
    }
    __syncthreads();
    const uint64_t dense = dense_lds;
    // buckets: 0 = dense slots only, 1 + s = first sparse virtual slot s; -1 = no row.
    // A histogram, its exclusive scan, then a position per row from the
    // bucket's cursor.  The order inside a bucket is whatever the atomics
    // give: every row is accumulated over its virtual slots in ascending
    // order whichever block it lands in, so results do not depend on it.
    int bkt[RPT];
#pragma unroll
    for (int rr = 0; rr < RPT; ++rr) {
      const int t = tid + rr * kDgradThreads;
      const uint64_t key = mrow[rr] & ~dense;
      bkt[rr] = t >= nrows ? -1 : (key ? 1 + __builtin_ctzll(key) : 0);
      if (bkt[rr] >= 0) atomicAdd(&hist[bkt[rr]], 1);
    }
    __syncthreads();
    if (wave == 0) {  // exclusive scan of NBK <= 128 counts, two per lane
      const int c0 = 2 * lane < NBK ? hist[2 * lane] : 0;
      const int c1 = 2 * lane + 1 < NBK ? hist[2 * lane + 1] : 0;
      const int local = c0 + c1;
      int inc = local;
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) {
        const int y = __shfl_up(inc, d, 64);
        if (lane >= d) inc += y;
      }
      const int run = inc - local;
      if (2 * lane < NBK) hist[2 * lane] = run;
      if (2 * lane + 1 < NBK) hist[2 * lane + 1] = run + c0;
    }
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < RPT; ++rr) {
      if (bkt[rr] >= 0) {
        const int pos = atomicAdd(&hist[bkt[rr]], 1);
        perm[pos] = tid + rr * kDgradThreads;
        if (mrow[rr]) atomicOr(reinterpret_cast<unsigned long long*>(&blkmask[pos >> 4]),
                               (unsigned long long)mrow[rr]);
      }
    }
    __syncthreads();
  }

  const __amdgpu_buffer_rsrc_t z_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<unsigned char*>(dZ), (short)0, (int)(n * Cout * E), kBufferWord3);
  const uint32_t row_bytes = (uint32_t)Cout * E;
  unsigned char* my = scratch + wave * 16 * WROW;
  // the row of the workgroup at sorted position p
  auto row_at = [&](int p) -> int { return TBL ? perm[p] : p; };

  struct Job {
    int blk;    // block, or -1 past the end
    int s;      // virtual slot, or -1 for a block without any
    bool last;  // last job of its block
  };
  // the wavefront's job sequence, generated block by block from the block
  // masks in LDS (wave-uniform state, no memory loads)
  int cur_blk = wave - kWaves;
  uint64_t rest = 0;
  auto next_job = [&]() -> Job {
    if (rest == 0) {
      cur_blk += kWaves;
      if (cur_blk * 16 >= nrows) return Job{-1, -1, true};
      const uint64_t m = TBL ? blkmask[cur_blk] : 1ull;
      if (m == 0) return Job{cur_blk, -1, true};
      rest = m;
    }
    const int sl = __builtin_ctzll(rest);
    rest &= rest - 1;
    return Job{cur_blk, sl, rest == 0};
  };
  struct Frags {
    i32x4 v[KSM];
  };
  // a job's source row (one lane per row), loaded ahead of its data; the
  // load is issued on every path (a clamped address when there is none) and
  // its value is only looked at when the data loads go out
  auto live_of = [&](const Job& jb) -> bool {
    return jb.blk >= 0 && jb.s >= 0 && jb.blk * 16 + l16 < nrows;
  };
  auto load_src = [&](const Job& jb, bool live) -> int32_t {
    const int64_t r = row0 + (live ? row_at(jb.blk * 16 + l16) : 0);
    if (!TBL) return (int32_t)r;
    return table_t[(live ? (int64_t)jb.s * n : 0) + r];
  };
  auto issue = [&](int32_t raw, bool live, Frags& f) {
    const int32_t src = live ? raw : -1;
    const uint32_t off = src >= 0 ? (uint32_t)src * row_bytes + (uint32_t)g * 16u : kOutOfRange;
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks)
      f.v[ks] = __builtin_bit_cast(
          i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                     z_rsrc, (ks < KS && ks * KW + (KW / 4) * g < Cout) ? off + (uint32_t)ks * 64u
                                                                         : kOutOfRange,
                     0, 0));
  };
  f32x4 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto compute = [&](const Job& jb, const Frags& f) {
    if (jb.blk < 0 || jb.s < 0) return;
    const int j = TBL ? slot_lds[jb.s] : 0;
#pragma unroll
    for (int ks = 0; ks < KSM; ++ks) {
      if (ks < KS) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const i32x4 bw = *reinterpret_cast<const i32x4*>(
              wl + ((size_t)((j * KS + ks) * NCB + cb) * 64 + lane) * 16);
          if constexpr (BF16) {
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, f.v[ks]),
                                                             __builtin_bit_cast(bf16x8, bw),
                                                             acc[cb], 0, 0, 0);
          } else {
            // lane group g holds reduction entries 4 g .. 4 g + 3 of the
            // k-step on both sides; MFMA s contracts component s
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2)
              acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(f.v[ks][s2]),
                                                             __int_as_float(bw[s2]), acc[cb], 0,
                                                             0, 0);
          }
        }
      }
    }
  };
  auto epilogue = [&](int blk) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      if constexpr (BF16) {
        // hardware round-to-nearest-even conversion, two rows per instruction
#pragma unroll
        for (int q = 0; q < 4; q += 2) {
          const bf16x2 h = __builtin_convertvector(f32x2{acc[cb][q], acc[cb][q + 1]}, bf16x2);
          *reinterpret_cast<__bf16*>(my + (4 * g + q) * WROW + (cb * 16 + l16) * 2) = h[0];
          *reinterpret_cast<__bf16*>(my + (4 * g + q + 1) * WROW + (cb * 16 + l16) * 2) = h[1];
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q)
          *reinterpret_cast<float*>(my + (4 * g + q) * WROW + (cb * 16 + l16) * 4) = acc[cb][q];
      }
      acc[cb] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    constexpr int VPRW = WS * E / 16;
#pragma unroll
    for (int idx0 = 0; idx0 < 16 * VPRW; idx0 += 64) {
      const int idx = idx0 + lane;
      const int rr = idx / VPRW, q = idx % VPRW;
      const int c = n0 + q * (16 / E);
      if (idx < 16 * VPRW && blk * 16 + rr < nrows && c < Cin) {
        const int64_t row = row0 + row_at(blk * 16 + rr);
        *reinterpret_cast<i32x4*>(dS + (row * Cin + c) * E) =
            *reinterpret_cast<const i32x4*>(my + rr * WROW + q * 16);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  };

  // Ring of D = DA + DS jobs in sequence order: slot u holds job t D + u.
  // Processing job k issues the data loads of job k + DA (its source row was
  // loaded DS jobs earlier) and takes job k + D, whose source load it issues.
  Job jobs[D];
  int32_t srcv[D];
  bool live[D];
  Frags fr[D];
#pragma unroll
  for (int u = 0; u < D; ++u) {
    jobs[u] = next_job();
    live[u] = live_of(jobs[u]);
    srcv[u] = load_src(jobs[u], live[u]);
  }
#pragma unroll
  for (int u = 0; u < DA; ++u) issue(srcv[u], live[u], fr[u]);
  while (jobs[0].blk >= 0) {
#pragma unroll
    for (int u = 0; u < D; ++u) {
      compute(jobs[u], fr[u]);
      if (jobs[u].blk >= 0 && jobs[u].last) epilogue(jobs[u].blk);
      issue(srcv[(u + DA) % D], live[(u + DA) % D], fr[(u + DA) % D]);
      jobs[u] = next_job();
      live[u] = live_of(jobs[u]);
      srcv[u] = load_src(jobs[u], live[u]);
    }
  }
}

}  // namespace

// ---------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

unsigned grid_for(int64_t n) { return (unsigned)std::max<int64_t>(1, (n + kThreads - 1) / kThreads); }

// column slice of the dgrad kernel: the widest of 128 / 64 / 32 / 16 input
// channels (not above Cin) whose weight fragments, scratch and sort arrays
// fit in LDS (a workgroup of eight wavefronts keeps two per SIMD)
size_t dgrad_lds(int ws, int32_t Kw, int32_t Cout, int e) {
  const int kw = e == 2 ? 32 : 16;
  const int KS = (Cout + kw - 1) / kw;
  return (size_t)Kw * KS * (ws / 16) * 1024 + (kDgradThreads / 64) * 16 * (ws * e + 16) +
         kDgradMaxRows / 16 * sizeof(uint64_t) + kDgradMaxRows * sizeof(int32_t) +
         (size_t)(kMaxVirtualSlots + 1) * sizeof(int32_t);
}

int dgrad_ws(int32_t Kw, int32_t Cin, int32_t Cout, int e) {
  for (int ws = 128; ws >= 16; ws /= 2) {
    if (ws > Cin && ws > 16) continue;
    if (dgrad_lds(ws, Kw, Cout, e) <= (size_t)kDgradLds) return ws;
  }
  return 0;
}

template <int WS, int KSM, bool TBL, bool BF16>
hipError_t launch_dgrad_ws(const void* dZ, const void* W, const int32_t* table_t,
                           const uint64_t* row_slots, const int32_t* slot_of, int64_t n,
                           int32_t Kw, int32_t Cin, int32_t Cout, void* dS, hipStream_t stream) {
  auto kern = dgrad_kernel<WS, KSM, TBL, BF16>;
  const size_t lds = dgrad_lds(WS, Kw, Cout, BF16 ? 2 : 4);
  // allow the large dynamic LDS allocation (up to kDgradLds); once per instantiation
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [&] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, kDgradLds);
  });
  if (attr_err != hipSuccess) return attr_err;
  const int slices = (Cin + WS - 1) / WS;
  // one wave of workgroups: as many row groups as the CUs hold workgroups
  // (all slices), whole 16-row blocks, 64 to kDgradMaxRows rows each; past
  // that many rows, more groups of the largest size
  const int64_t per_cu = std::max<int64_t>(1, (int64_t)(160 * 1024) / (int64_t)(lds + 1024));
  const int64_t groups = std::max<int64_t>(1, 256 * per_cu / slices);
  int64_t R = (n + groups - 1) / groups;
  R = std::min<int64_t>(kDgradMaxRows, std::max<int64_t>(64, (R + 15) / 16 * 16));
  const unsigned gx = (unsigned)((n + R - 1) / R);
  hipLaunchKernelGGL(kern, dim3(gx, (unsigned)slices), dim3(kDgradThreads), lds, stream,
                     static_cast<const unsigned char*>(dZ), static_cast<const unsigned char*>(W),
                     table_t, row_slots, slot_of, n, Kw, Cin, Cout, (int32_t)R,
                     static_cast<unsigned char*>(dS));
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// the bf16 linear layer's backward in one pass over the rows
// ---------------------------------------------------------------------------

// C_in, C_out in {64, 128}.  Workgroup w takes rows [w L, w L + L), 32 rows
// per step, with the loads of the next kLinRing - 1 steps in flight in
// registers.  Per step:
//   * dZ = dY (.) [Y > 0] of the step's rows, formed from the loaded dY and Y
//     vectors (rows past n read as zeros), its column sums added per thread
//     in fp32 (the bias gradient), and staged in LDS with the S rows;
//   * dS rows = dZ W^T: A fragments are 16 contiguous bytes of a dZ row, the
//     B fragments of W^T (W[c][o .. o + 7], 16 contiguous bytes) stay in
//     registers for the whole launch; the rounded rows go out as whole
//     16-byte vectors through an LDS tile;
//   * the workgroup's partial dW += S^T dZ over the step's 32 rows, both
//     operands read with transposing LDS reads (wgrad_tile's scheme).
// At the end the partial tile (fp32, in wgrad_tile's chunk layout, chunk w)
// and the column sums (colpart[w]) go to the workspace; wgrad_reduce_kernel
// then sums them over the chunks in a fixed order.
constexpr int kLinThreads = 512;
constexpr int kLinRing = 3;
template <int CI, int CO>
__global__ __launch_bounds__(kLinThreads) void linear_bwd_fused_kernel(
    const __bf16* __restrict__ S, const __bf16* __restrict__ W, const __bf16* __restrict__ Y,
    const __bf16* __restrict__ dY, int64_t n, int32_t L, int act, int32_t T,
    __bf16* __restrict__ dS, float* __restrict__ part, float* __restrict__ colpart) {
  constexpr int R = 32;
  constexpr int NCI = CI / 16, NCO = CO / 16, KSO = CO / 32;
  constexpr int ROWI = CI * 2 + 16, ROWO = CO * 2 + 16;  // padded LDS rows
  constexpr int VPI = CI / 8, VPO = CO / 8;              // 16-byte vectors per row
  constexpr int NVI = (R * VPI + kLinThreads - 1) / kLinThreads;
  constexpr int NVO = (R * VPO + kLinThreads - 1) / kLinThreads;
  // dgrad: 2 row blocks x NCI column blocks, DCB column blocks per wavefront
  constexpr int DCB = NCI / 4;
  // wgrad: wavefront (wa, wb) of 2 x 4 takes NBA x NBB blocks of 16 x 16
  constexpr int NBA = NCI / 2, NBB = NCO / 4;
  static_assert((CI == 64 || CI == 128) && (CO == 64 || CO == 128), "C_in, C_out in {64, 128}");
  static_assert(kLinThreads % VPI == 0 && kLinThreads % VPO == 0, "column of a thread");
  __shared__ __attribute__((aligned(16))) unsigned char st_s[R * ROWI];
  __shared__ __attribute__((aligned(16))) unsigned char st_z[R * ROWO];
  __shared__ __attribute__((aligned(16))) unsigned char st_d[R * ROWI];
  __shared__ float csum[kLinThreads * 8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int g = lane >> 4, l16 = lane & 15;
  const int64_t row0 = (int64_t)blockIdx.x * L;
  const int rows = (int)min((int64_t)L, n - row0);
  const int steps = (rows + R - 1) / R;

  // B fragments of W^T for this wavefront's dgrad blocks: row block rb,
  // column blocks cb0 .. cb0 + DCB - 1
  // (each output optional: W is read only for dS, S only for dW)
  const bool do_ds = dS != nullptr, do_dw = part != nullptr;
  const int rb = wave & 1, cb0 = (wave >> 1) * DCB;
  bf16x8 wt[DCB][KSO];
#pragma unroll
  for (int x = 0; x < DCB; ++x)
#pragma unroll
    for (int ks = 0; ks < KSO; ++ks)
      wt[x][ks] = do_ds ? *reinterpret_cast<const bf16x8*>(
                              W + (int64_t)((cb0 + x) * 16 + l16) * CO + ks * 32 + 8 * g)
                        : bf16x8{};

  struct Regs {
    i32x4 dy[NVO], y[NVO], s[NVI];
  };
  // the loads of step st (rows past n, or steps past the last, clamped to
  // row 0 of the workgroup and zeroed when used)
  auto load = [&](int st, Regs& r) {
#pragma unroll
    for (int u = 0; u < NVO; ++u) {
      const int e = tid + u * kLinThreads;
      const int rr = e / VPO, q = e % VPO;
      const int64_t row = row0 + (int64_t)st * R + rr;
      const int64_t idx = (row < n && e < R * VPO ? row : row0) * CO + q * 8;
      r.dy[u] = *reinterpret_cast<const i32x4*>(dY + idx);
      r.y[u] = *reinterpret_cast<const i32x4*>(Y + idx);  // Y = dY when there is no ReLU
    }
#pragma unroll
    for (int u = 0; u < NVI; ++u) {
      const int e = tid + u * kLinThreads;
      const int rr = e / VPI, q = e % VPI;
      const int64_t row = row0 + (int64_t)st * R + rr;
      const int64_t idx = (row < n && e < R * VPI ? row : row0) * CI + q * 8;
      r.s[u] = do_dw ? *reinterpret_cast<const i32x4*>(S + idx) : i32x4{0, 0, 0, 0};
    }
  };

  // transposing read of 32 rows x 16 columns (block cb) of a staged tile
  auto frag = [&](const unsigned char* base, int row_bytes, int cb) -> bf16x8 {
    const unsigned char* p0 = base + (8 * g + (l16 >> 2)) * row_bytes + cb * 32 + 8 * (l16 & 3);
    const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0)));
    const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
        (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0 + 4 * row_bytes)));
    return bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  };

  const int wa = wave >> 2, wb = wave & 3;
  f32x4 wacc[NBA][NBB];
#pragma unroll
  for (int x = 0; x < NBA; ++x)
#pragma unroll
    for (int y = 0; y < NBB; ++y) wacc[x][y] = f32x4{0.f, 0.f, 0.f, 0.f};
  float cs[8];
#pragma unroll
  for (int k = 0; k < 8; ++k) cs[k] = 0.f;

  auto body = [&](int st, Regs& r) {
    if (st >= steps) return;
    const int64_t rbase = row0 + (int64_t)st * R;
    // dZ and its column sums, staged with the S rows
#pragma unroll
    for (int u = 0; u < NVO; ++u) {
      const int e = tid + u * kLinThreads;
      const int rr = e / VPO, q = e % VPO;
      const bool live = e < R * VPO && rbase + rr < n;
      i32x4 z = r.dy[u];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const uint32_t gw = live ? (uint32_t)z[w] : 0u;
        const uint32_t yv = (uint32_t)r.y[u][w];
        const uint32_t lo = (!act || bf16_bits_to_f32(yv & 0xFFFFu) > 0.f) ? (gw & 0xFFFFu) : 0u;
        const uint32_t hi = (!act || bf16_bits_to_f32(yv >> 16) > 0.f) ? (gw & 0xFFFF0000u) : 0u;
        z[w] = (int)(lo | hi);
        cs[2 * w] += bf16_bits_to_f32(lo);
        cs[2 * w + 1] += bf16_bits_to_f32(hi >> 16);
      }
      if (e < R * VPO) *reinterpret_cast<i32x4*>(st_z + rr * ROWO + q * 16) = z;
    }
#pragma unroll
    for (int u = 0; u < NVI; ++u) {
      const int e = tid + u * kLinThreads;
      const int rr = e / VPI, q = e % VPI;
      const bool live = e < R * VPI && rbase + rr < n;
      if (e < R * VPI)
        *reinterpret_cast<i32x4*>(st_s + rr * ROWI + q * 16) = live ? r.s[u] : i32x4{0, 0, 0, 0};
    }
    __syncthreads();
    // the registers are free: the loads of step st + kLinRing
    load(st + kLinRing, r);
    // dS rows of the step (zeros, never stored, without dS)
    f32x4 dacc[DCB];
#pragma unroll
    for (int x = 0; x < DCB; ++x) dacc[x] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KSO; ++ks) {
      const bf16x8 a = *reinterpret_cast<const bf16x8*>(st_z + (16 * rb + l16) * ROWO +
                                                        (32 * ks + 8 * g) * 2);
#pragma unroll
      for (int x = 0; x < DCB; ++x)
        dacc[x] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, wt[x][ks], dacc[x], 0, 0, 0);
    }
    // partial dW over the step's rows (always run: S reads as zeros without
    // dW, and no branch separates the dgrad MFMAs above from the reads of
    // their results below)
    {
      bf16x8 fa[NBA], fb[NBB];
#pragma unroll
      for (int x = 0; x < NBA; ++x) fa[x] = frag(st_s, ROWI, wa * NBA + x);
#pragma unroll
      for (int y = 0; y < NBB; ++y) fb[y] = frag(st_z, ROWO, wb * NBB + y);
#pragma unroll
      for (int x = 0; x < NBA; ++x)
#pragma unroll
        for (int y = 0; y < NBB; ++y)
          wacc[x][y] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fa[x], fb[y], wacc[x][y], 0, 0, 0);
    }
    // dS tile: rows 16 rb + 4 g + i, columns 16 (cb0 + x) + l16, rounded to
    // nearest even by the hardware conversion
#pragma unroll
    for (int x = 0; x < DCB; ++x) {
      unsigned char* pp = st_d + (16 * rb + 4 * g) * ROWI + ((cb0 + x) * 16 + l16) * 2;
#pragma unroll
      for (int i = 0; i < 4; i += 2) {
        const bf16x2 h = __builtin_convertvector(f32x2{dacc[x][i], dacc[x][i + 1]}, bf16x2);
        *reinterpret_cast<__bf16*>(pp + i * ROWI) = h[0];
        *reinterpret_cast<__bf16*>(pp + (i + 1) * ROWI) = h[1];
      }
    }
    __syncthreads();
    if (do_ds) {
#pragma unroll
      for (int u = 0; u < NVI; ++u) {
        const int e = tid + u * kLinThreads;
        const int rr = e / VPI, q = e % VPI;
        if (e < R * VPI && rbase + rr < n)
          *reinterpret_cast<i32x4*>(dS + (rbase + rr) * CI + q * 8) =
              *reinterpret_cast<const i32x4*>(st_d + rr * ROWI + q * 16);
      }
    }
  };

  Regs r0, r1, r2;
  static_assert(kLinRing == 3, "three register sets");
  load(0, r0);
  load(1, r1);
  load(2, r2);
  for (int st = 0; st < steps; st += kLinRing) {
    body(st, r0);
    body(st + 1, r1);
    body(st + 2, r2);
  }

  // partial tile of chunk w (wgrad_tile's layout: tile (ta, tb) of T x T)
  if (part != nullptr) {
    const int tB = CO / T;
    const int tiles = (CI / T) * tB;
#pragma unroll
    for (int x = 0; x < NBA; ++x)
#pragma unroll
      for (int y = 0; y < NBB; ++y)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int c = (wa * NBA + x) * 16 + 4 * g + i;
          const int o = (wb * NBB + y) * 16 + l16;
          const int ta = c / T, tb = o / T;
          part[((int64_t)blockIdx.x * tiles + ta * tB + tb) * T * T + (c - ta * T) * T +
               (o - tb * T)] = wacc[x][y][i];
        }
  }
  // column sums: threads with the same 16-byte column vector, in thread order
  if (colpart != nullptr) {
#pragma unroll
    for (int k = 0; k < 8; ++k) csum[tid * 8 + k] = cs[k];
    __syncthreads();
    for (int c = tid; c < CO; c += kLinThreads) {
      const int q = c / 8, k = c % 8;
      float t = 0.f;
      for (int th = q; th < kLinThreads; th += VPO) t += csum[th * 8 + k];
      colpart[(int64_t)blockIdx.x * CO + c] = t;
    }
  }
}

struct LinBwdArgs {
  const __bf16 *S, *W, *Y, *dY;
  int64_t n;
  int32_t L;
  int act;
  int32_t T;
  __bf16* dS;
  float *part, *colpart;
};

template <int CI, int CO>
void launch_linear_bwd_fused(const LinBwdArgs& a, unsigned grid, hipStream_t stream) {
  hipLaunchKernelGGL((linear_bwd_fused_kernel<CI, CO>), dim3(grid), dim3(kLinThreads), 0, stream,
                     a.S, a.W, a.Y, a.dY, a.n, a.L, a.act, a.T, a.dS, a.part, a.colpart);
}

template <int WS, bool BF16>
hipError_t launch_dgrad_k(const void* dZ, const void* W, const int32_t* table_t,
                          const uint64_t* row_slots, const int32_t* slot_of, int64_t n,
                          int32_t Kw, int32_t Cin, int32_t Cout, void* dS, hipStream_t stream) {
  const bool tbl = table_t != nullptr;
  const int ks = BF16 ? (Cout + 31) / 32 : (Cout + 15) / 16;  // k-steps: at most 8 / 16
  if (ks <= 4)
    return tbl ? launch_dgrad_ws<WS, 4, true, BF16>(dZ, W, table_t, row_slots, slot_of, n, Kw,
                                                    Cin, Cout, dS, stream)
               : launch_dgrad_ws<WS, 4, false, BF16>(dZ, W, table_t, row_slots, slot_of, n, Kw,
                                                     Cin, Cout, dS, stream);
  if (ks <= 8)
    return tbl ? launch_dgrad_ws<WS, 8, true, BF16>(dZ, W, table_t, row_slots, slot_of, n, Kw,
                                                    Cin, Cout, dS, stream)
               : launch_dgrad_ws<WS, 8, false, BF16>(dZ, W, table_t, row_slots, slot_of, n, Kw,
                                                     Cin, Cout, dS, stream);
  if constexpr (!BF16)
    return tbl ? launch_dgrad_ws<WS, 16, true, false>(dZ, W, table_t, row_slots, slot_of, n, Kw,
                                                      Cin, Cout, dS, stream)
               : launch_dgrad_ws<WS, 16, false, false>(dZ, W, table_t, row_slots, slot_of, n,
                                                       Kw, Cin, Cout, dS, stream);
  return hipErrorInvalidValue;
}

}  // namespace

int backward_dgrad_supported(int32_t Kw, int32_t Cin, int32_t Cout, int is_bf16) {
  return Cout <= 256 && Kw <= kMaxSlotsBwd && dgrad_ws(Kw, Cin, Cout, is_bf16 ? 2 : 4) > 0;
}

void backward_plan(int64_t n, int32_t K, int32_t Cin, int32_t Cout, int is_bf16, int conv,
                   BwdPlan* p) {
  const int e = is_bf16 ? 2 : 4;
  p->T = (is_bf16 && Cin % 128 == 0 && Cout % 128 == 0) ? 128 : 64;
  p->tiles = ((Cin + p->T - 1) / p->T) * ((Cout + p->T - 1) / p->T);
  const int64_t per = conv ? (int64_t)K * ((n + 255) / 256) : (n + 255) / 256;
  p->L = per > 8192 ? 512 : 256;
  p->max_chunks = conv ? (int64_t)K * ((n + p->L - 1) / p->L) : (n + p->L - 1) / p->L;
  p->splits = (int)std::min<int64_t>(2048, std::max<int64_t>(1, (n + 63) / 64));
  p->rps = std::max<int64_t>(1, (n + p->splits - 1) / p->splits);
  size_t o = 0;
  p->off_dz = o;
  o += align256((size_t)n * Cout * e);
  p->off_colpart = o;
  o += align256((size_t)p->splits * Cout * sizeof(float));
  const int64_t kn = conv ? (int64_t)K * n : 0;
  p->off_pairs = o;
  o += align256((size_t)kn * 8);
  p->off_rowptr = o;
  o += align256((size_t)(K + 1) * 4);
  p->off_mask = o;  // the pair build's own workspace
  o += conv ? slot_pairs_ws_bytes(n, K) : 0;
  // partial tiles: sized for chunks of 256 rows whatever L is, so the
  // workspace never shrinks as n grows
  const int64_t cap_chunks = conv ? (int64_t)K * ((n + 255) / 256) : (n + 255) / 256;
  p->off_part = o;
  o += align256((size_t)std::max<int64_t>(cap_chunks, p->max_chunks) * p->tiles * p->T * p->T *
                sizeof(float));
  p->total = o;
}

size_t transpose_neighbors_ws_bytes(int32_t V, int32_t K) {
  return align256((size_t)V * K * 4) * 2 + align256((size_t)(K + 1) * 4);
}

hipError_t launch_transpose_neighbors(const int32_t* nbr, int32_t V, int32_t K, int32_t* nbr_t,
                                      int32_t* slot_of, int32_t* off_dev, void* ws,
                                      hipStream_t stream) {
  unsigned char* w = static_cast<unsigned char*>(ws);
  int32_t* cnt = reinterpret_cast<int32_t*>(w);
  int32_t* cur = reinterpret_cast<int32_t*>(w + align256((size_t)V * K * 4));
  const int64_t vk = (int64_t)V * K;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(std::min<unsigned>(grid_for(vk), 4096)), dim3(kThreads),
                     0, stream, cnt, vk, 0);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(std::min<unsigned>(grid_for(vk), 4096)), dim3(kThreads),
                     0, stream, cur, vk, 0);
  const int64_t cap = (int64_t)V * kMaxVirtualSlots;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(std::min<unsigned>(grid_for(cap), 4096)),
                     dim3(kThreads), 0, stream, nbr_t, cap, -1);
  hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(kThreads), 0, stream, slot_of,
                     (int64_t)kMaxVirtualSlots, -1);
  hipLaunchKernelGGL(tv_count_kernel, dim3(grid_for(vk)), dim3(kThreads), 0, stream, nbr, V, K, cnt);
  hipLaunchKernelGGL(tv_layout_kernel, dim3(1), dim3(kThreads), 0, stream, cnt, V, K, off_dev,
                     slot_of, (int32_t)kMaxVirtualSlots);
  hipLaunchKernelGGL(tv_fill_kernel, dim3(grid_for(vk)), dim3(kThreads), 0, stream, nbr, V, K,
                     off_dev, cur, nbr_t, (int32_t)kMaxVirtualSlots);
  hipLaunchKernelGGL(tv_sort_kernel, dim3(grid_for(vk)), dim3(kThreads), 0, stream, cnt, V, K,
                     off_dev, nbr_t, (int32_t)kMaxVirtualSlots);
  return hipGetLastError();
}

hipError_t launch_transposed_table(const int32_t* coords, const int32_t* inv, int64_t n, int32_t B,
                                   int32_t V, const int32_t* nbr_t, int32_t Kt, int32_t* table_t,
                                   uint64_t* row_slots, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(tt_kernel, dim3(grid_for(4 * n)), dim3(kThreads), 0, stream,
                     reinterpret_cast<const int2*>(coords), inv, n, B, V, nbr_t, Kt, table_t,
                     row_slots);
  return hipGetLastError();
}

hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t stream) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(fill_i32_kernel, dim3(std::min<unsigned>(grid_for(n), 4096)), dim3(kThreads),
                     0, stream, p, n, v);
  return hipGetLastError();
}

size_t slot_pairs_ws_bytes(int64_t n, int32_t K) {
  int32_t nb = 0;
  int64_t per_block = 0;
  const int64_t kn = (int64_t)K * n;
  if (kn > 0) compact_plan(kn, &nb, &per_block);
  return align256((size_t)kn) + align256((size_t)kn * 4) + align256(16) + align256((size_t)nb * 4);
}

// Pair lists of an active set: (slot j, row i) for every table[j][i] >= 0,
// slot-major with rows ascending (a compaction of the [K][n] presence
// mask), and the slot offsets pair_ptr[K + 1].  ws: slot_pairs_ws_bytes.
hipError_t launch_slot_pairs(const int32_t* table, int64_t n, int32_t K, int32_t* pairs,
                             int32_t* pair_ptr, void* ws, hipStream_t stream) {
  unsigned char* w = static_cast<unsigned char*>(ws);
  const int64_t kn = (int64_t)K * n;
  uint8_t* mask = w;
  int32_t* inv_p = reinterpret_cast<int32_t*>(w + align256((size_t)kn));
  int32_t* nact = reinterpret_cast<int32_t*>(w + align256((size_t)kn) + align256((size_t)kn * 4));
  int32_t* bc = nact + 64;
  hipLaunchKernelGGL(presence_kernel, dim3(std::min<unsigned>(grid_for(kn), 8192)), dim3(kThreads),
                     0, stream, table, kn, mask);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_compact(mask, K, (int32_t)n, pairs, inv_p, pair_ptr, nact, nullptr, kn, bc,
                        stream);
}

hipError_t launch_layer_backward(int conv, const void* S, const int32_t* table,
                                 const int32_t* pairs, const int32_t* pair_ptr,
                                 const int32_t* table_t, const uint64_t* row_slots,
                                 const int32_t* slot_of, const void* W, const void* Y,
                                 const void* dY, int64_t n, int32_t K, int32_t Cin, int32_t Cout,
                                 int is_bf16, int act, void* dS, float* dW, float* db, void* ws,
                                 hipStream_t stream) {
  BwdPlan pl;
  backward_plan(n, K, Cin, Cout, is_bf16, conv, &pl);
  unsigned char* w = static_cast<unsigned char*>(ws);
  const int Kw = conv ? K : 1;
  if (n == 0) {  // no rows: zero weight and bias gradients
    if (dW != nullptr)
      hipLaunchKernelGGL(fill_i32_kernel, dim3(64), dim3(kThreads), 0, stream,
                         reinterpret_cast<int32_t*>(dW), (int64_t)Kw * Cin * Cout, 0);
    if (db != nullptr)
      hipLaunchKernelGGL(fill_i32_kernel, dim3(1), dim3(kThreads), 0, stream,
                         reinterpret_cast<int32_t*>(db), (int64_t)Cout, 0);
    return hipGetLastError();
  }
  // the bf16 linear layer of 64 or 128 channels: one pass over the rows,
  // then the reduction of its per-workgroup partials
  if (!conv && is_bf16 && (Cin == 64 || Cin == 128) && (Cout == 64 || Cout == 128)) {
    int dev = 0, cus = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e != hipSuccess) return e;
    // about one workgroup per CU, at least 256 rows each (the workspace holds
    // partials for chunks of 256 rows)
    int64_t L = (n + cus - 1) / cus;
    L = std::max<int64_t>(256, (L + 31) / 32 * 32);
    const int64_t G = (n + L - 1) / L;
    float* part = dW != nullptr ? reinterpret_cast<float*>(w + pl.off_part) : nullptr;
    float* colpart = db != nullptr ? reinterpret_cast<float*>(w + pl.off_colpart) : nullptr;
    const LinBwdArgs la{static_cast<const __bf16*>(S), static_cast<const __bf16*>(W),
                        static_cast<const __bf16*>(act ? Y : dY), static_cast<const __bf16*>(dY),
                        n, (int32_t)L, act, pl.T, static_cast<__bf16*>(dS), part, colpart};
    if (Cin == 128) {
      if (Cout == 128) launch_linear_bwd_fused<128, 128>(la, (unsigned)G, stream);
      else launch_linear_bwd_fused<128, 64>(la, (unsigned)G, stream);
    } else {
      if (Cout == 128) launch_linear_bwd_fused<64, 128>(la, (unsigned)G, stream);
      else launch_linear_bwd_fused<64, 64>(la, (unsigned)G, stream);
    }
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (dW != nullptr) {
      const dim3 rg((unsigned)(pl.tiles + (db != nullptr ? 1 : 0)), (unsigned)(pl.T * pl.T / 32));
      if (pl.T == 128)
        hipLaunchKernelGGL((wgrad_reduce_kernel<128, 32>), rg, dim3(32 * 32), 0, stream, part,
                           nullptr, (int32_t)L, Cin, Cout, 1, (int32_t)G, dW, colpart, (int32_t)G,
                           db);
      else
        hipLaunchKernelGGL((wgrad_reduce_kernel<64, 32>), rg, dim3(32 * 32), 0, stream, part,
                           nullptr, (int32_t)L, Cin, Cout, 1, (int32_t)G, dW, colpart, (int32_t)G,
                           db);
    } else if (db != nullptr) {
      hipLaunchKernelGGL(colsum_kernel, dim3((Cout + 7) / 8), dim3(kThreads), 0, stream, colpart,
                         (int)G, Cout, db);
    }
    return hipGetLastError();
  }
  // dZ (through the ReLU) and the bias gradient
  const void* dZ = dY;
  if (act || db != nullptr) {
    float* colpart = reinterpret_cast<float*>(w + pl.off_colpart);
    void* dz_out = act ? static_cast<void*>(w + pl.off_dz) : nullptr;
    if (is_bf16)
      hipLaunchKernelGGL(relu_bwd_kernel<true>, dim3(pl.splits), dim3(kThreads), 0, stream,
                         static_cast<const i32x4*>(dY), static_cast<const i32x4*>(Y), n, Cout,
                         act, pl.rps, static_cast<i32x4*>(dz_out), colpart);
    else
      hipLaunchKernelGGL(relu_bwd_kernel<false>, dim3(pl.splits), dim3(kThreads), 0, stream,
                         static_cast<const i32x4*>(dY), static_cast<const i32x4*>(Y), n, Cout,
                         act, pl.rps, static_cast<i32x4*>(dz_out), colpart);
    if (act) dZ = dz_out;
    // the bias gradient's column sums: in the weight gradient's reduction
    // launch when there is one, else on their own
    if (db != nullptr && dW == nullptr)
      hipLaunchKernelGGL(colsum_kernel, dim3((Cout + 7) / 8), dim3(kThreads), 0, stream, colpart,
                         pl.splits, Cout, db);
  }
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  // weight gradient
  if (dW != nullptr) {
    float* part = reinterpret_cast<float*>(w + pl.off_part);
    const int2* pr = nullptr;
    const int32_t* rp = nullptr;
    if (conv) {
      if (pairs != nullptr) {
        pr = reinterpret_cast<const int2*>(pairs);
        rp = pair_ptr;
      } else {
        int32_t* prw = reinterpret_cast<int32_t*>(w + pl.off_pairs);
        int32_t* rpw = reinterpret_cast<int32_t*>(w + pl.off_rowptr);
        err = launch_slot_pairs(table, n, K, prw, rpw, w + pl.off_mask, stream);
        if (err != hipSuccess) return err;
        pr = reinterpret_cast<const int2*>(prw);
        rp = rpw;
      }
    }
    const unsigned gt = (unsigned)(pl.max_chunks * pl.tiles);
    if (!is_bf16)
      hipLaunchKernelGGL((wgrad_tile_f32_kernel<64, 32>), dim3(gt), dim3(kThreads), 0, stream,
                         static_cast<const float*>(S), static_cast<const float*>(dZ), table, pr,
                         rp, Kw, n, pl.L, Cin, Cout, part);
    else if (pl.T == 128)
      hipLaunchKernelGGL((wgrad_tile_kernel<128, kWgradRows>), dim3(gt), dim3(kThreads), 0, stream,
                         static_cast<const __bf16*>(S), static_cast<const __bf16*>(dZ), table, pr,
                         rp, Kw, n, pl.L, Cin, Cout, part);
    else
      hipLaunchKernelGGL((wgrad_tile_kernel<64, kWgradRows>), dim3(gt), dim3(kThreads), 0, stream,
                         static_cast<const __bf16*>(S), static_cast<const __bf16*>(dZ), table, pr,
                         rp, Kw, n, pl.L, Cin, Cout, part);
    err = hipGetLastError();
    if (err != hipSuccess) return err;
    // one more column of workgroups reduces the bias gradient (T * T / 32 >= Cout / 32)
    const float* cp = db != nullptr ? reinterpret_cast<const float*>(w + pl.off_colpart) : nullptr;
    const dim3 rg((unsigned)(Kw * pl.tiles + (db != nullptr ? 1 : 0)),
                  (unsigned)(pl.T * pl.T / 32));
#define SHC_REDUCE(TT, GG)                                                                     \
  hipLaunchKernelGGL((wgrad_reduce_kernel<TT, GG>), rg, dim3(32 * GG), 0, stream, part, rp, pl.L, \
                     Cin, Cout, conv ? 0 : 1, (int32_t)pl.max_chunks, dW, cp, pl.splits, db)
    if (pl.T == 128) {
      if (conv) SHC_REDUCE(128, 8); else SHC_REDUCE(128, 32);
    } else {
      if (conv) SHC_REDUCE(64, 8); else SHC_REDUCE(64, 32);
    }
#undef SHC_REDUCE
    err = hipGetLastError();
    if (err != hipSuccess) return err;
  }
  // input gradient
  if (dS != nullptr) {
    const int wsl = dgrad_ws(Kw, Cin, Cout, is_bf16 ? 2 : 4);
    const int32_t* tt = conv ? table_t : nullptr;
    const uint64_t* rs = conv ? row_slots : nullptr;
    const int32_t* so = conv ? slot_of : nullptr;
    if (is_bf16) {
      switch (wsl) {
        case 128: err = launch_dgrad_k<128, true>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
        case 64: err = launch_dgrad_k<64, true>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
        case 32: err = launch_dgrad_k<32, true>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
        default: err = launch_dgrad_k<16, true>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
      }
    } else {
      switch (wsl) {
        case 128: err = launch_dgrad_k<128, false>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
        case 64: err = launch_dgrad_k<64, false>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
        case 32: err = launch_dgrad_k<32, false>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
        default: err = launch_dgrad_k<16, false>(dZ, W, tt, rs, so, n, Kw, Cin, Cout, dS, stream); break;
      }
    }
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

}  // namespace shc
