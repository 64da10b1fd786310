// Row movers of the sparse path: gather of the active rows (S' of Eq. 2),
// scatter back to the dense per-vertex layout, and the per-body max-pool.
//
// All three are HBM-bound copies/selections.  Rows are moved as 16-byte
// vectors: a block is a (tx, ty) grid of threads where tx threads cover one
// row (tx = vectors per row, capped at 256) and ty rows are in flight, so
// every wavefront issues contiguous 16-byte accesses along a row and no
// integer division is needed per element.
#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kThreads = 256;

struct RowShape {
  int vpr;  // 16-byte vectors per row
  int tx;   // threads per row
  int ty;   // rows per block
};

RowShape row_shape(int32_t row_bytes) {
  RowShape s;
  s.vpr = row_bytes / 16;
  s.tx = s.vpr < kThreads ? s.vpr : kThreads;
  s.ty = kThreads / s.tx;
  return s;
}

// Each thread moves vector q of kGatherRows rows (ty apart), issuing every
// coordinate load, then every row load, before the first store, so each
// thread keeps kGatherRows 16-byte loads in flight.  Rows past n_rows clamp to
// the last row (loaded, never stored); a coordinate outside [0,B)x[0,V)
// reads row 0 and stores zeros.
constexpr int kGatherRows = 4;

// MASK: 0 = plain rows; 1 / 2 = rows multiplied by a per-element 0/1 mask
// of bf16 / fp32 channels (8 / 4 mask bytes per 16-byte vector).  Coordinates
// name bodies in [0, B); body b reads input body b mod Bx (Bx = B but for
// several masks stacked as a batch axis).
template <int MASK>
__global__ __launch_bounds__(kThreads) void gather_kernel(const i32x4* __restrict__ x,
                                                          const uint8_t* __restrict__ me,
                                                          const int2* __restrict__ coords,
                                                          int64_t n_rows, int32_t B, int32_t Bx,
                                                          int32_t V, int vpr,
                                                          i32x4* __restrict__ S) {
  const int ty = blockDim.y;
  const int64_t i0 = (int64_t)blockIdx.x * kGatherRows * ty + threadIdx.y;
  int64_t src[kGatherRows];
  bool ok[kGatherRows];
#pragma unroll
  for (int k = 0; k < kGatherRows; ++k) {
    const int64_t i = min(i0 + (int64_t)k * ty, n_rows - 1);
    const int2 c = coords[i];
    ok[k] = c.x >= 0 && c.x < B && c.y >= 0 && c.y < V;
    const int bx = c.x < Bx ? c.x : c.x % Bx;
    src[k] = ok[k] ? ((int64_t)bx * V + c.y) * vpr : 0;
  }
  for (int q = threadIdx.x; q < vpr; q += blockDim.x) {
    i32x4 val[kGatherRows];
#pragma unroll
    for (int k = 0; k < kGatherRows; ++k) val[k] = __builtin_nontemporal_load(x + src[k] + q);
    if (MASK != 0) {
      constexpr int kPer = MASK == 1 ? 8 : 4;  // channels (mask bytes) per vector
#pragma unroll
      for (int k = 0; k < kGatherRows; ++k) {
        const uint8_t* mb = me + (src[k] + q) * kPer;  // element (row, channel) mask bytes
        uint64_t bytes = MASK == 1 ? *reinterpret_cast<const uint64_t*>(mb)
                                   : (uint64_t)*reinterpret_cast<const uint32_t*>(mb);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          uint32_t keep;
          if (MASK == 1) {
            keep = (((bytes >> (16 * e)) & 0xFFu) ? 0x0000FFFFu : 0u) |
                   (((bytes >> (16 * e + 8)) & 0xFFu) ? 0xFFFF0000u : 0u);
          } else {
            keep = ((bytes >> (8 * e)) & 0xFFu) ? 0xFFFFFFFFu : 0u;
          }
          val[k][e] &= (int)keep;
        }
      }
    }
#pragma unroll
    for (int k = 0; k < kGatherRows; ++k) {
      const int64_t i = i0 + (int64_t)k * ty;
      if (i < n_rows) S[i * vpr + q] = ok[k] ? val[k] : i32x4{0, 0, 0, 0};
    }
  }
}

// out[v] = op over k < kappa of Y[k * n_vec + v], per channel of 16-byte
// vector v (OP 0 sum, 1 mean, 2 max), accumulated in fp32 in k order.
template <int OP, bool BF16>
__global__ __launch_bounds__(kThreads) void combine_kernel(const i32x4* __restrict__ Y,
                                                           int32_t kappa, int64_t n_vec,
                                                           i32x4* __restrict__ out) {
  const int64_t v = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (v >= n_vec) return;
  constexpr int N = BF16 ? 8 : 4;
  float acc[N];
  auto widen = [&](const i32x4& w, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (BF16) {
        f[2 * e] = __int_as_float(w[e] << 16);
        f[2 * e + 1] = __int_as_float(w[e] & (int)0xFFFF0000);
      } else {
        f[e] = __int_as_float(w[e]);
      }
    }
  };
  widen(__builtin_nontemporal_load(Y + v), acc);
  for (int k = 1; k < kappa; ++k) {
    float f[N];
    widen(__builtin_nontemporal_load(Y + (int64_t)k * n_vec + v), f);
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = OP == 2 ? (f[e] > acc[e] ? f[e] : acc[e]) : acc[e] + f[e];
  }
  if (OP == 1)
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = acc[e] / (float)kappa;
  i32x4 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    if (BF16) {  // hardware round-to-nearest-even conversion, two channels at a time
      typedef float f2 __attribute__((ext_vector_type(2)));
      typedef __bf16 h2 __attribute__((ext_vector_type(2)));
      o[e] = __builtin_bit_cast(int, __builtin_convertvector(f2{acc[2 * e], acc[2 * e + 1]}, h2));
    } else {
      o[e] = __float_as_int(acc[e]);
    }
  }
  __builtin_nontemporal_store(o, out + v);
}

// m[b * V + v] = 1 when any of the C mask bytes of (b, v) is non-zero, else 0.
// tx lanes (a power of two <= 64) share a vertex, each ORing every tx-th of
// its C / 16 chunks, and a ballot over the wavefront ORs the vertex's lanes.
__global__ __launch_bounds__(kThreads) void row_activity_kernel(const i32x4* __restrict__ me,
                                                                int64_t n_vert, int vpr, int tx,
                                                                uint8_t* __restrict__ m) {
  const int lane = threadIdx.x & 63;
  const int64_t vert = ((int64_t)blockIdx.x * kThreads + threadIdx.x) / tx;
  const int sub = lane % tx;
  bool nz = false;
  if (vert < n_vert)
    for (int q = sub; q < vpr; q += tx) {
      const i32x4 w = __builtin_nontemporal_load(me + vert * vpr + q);
      nz |= (w[0] | w[1] | w[2] | w[3]) != 0;
    }
  const uint64_t bal = __ballot(nz);
  const int slot = lane / tx;
  const uint64_t lanes = (tx == 64 ? ~0ull : ((1ull << tx) - 1ull)) << (slot * tx);
  if (vert < n_vert && sub == 0) m[vert] = (bal & lanes) ? 1 : 0;
}

// D[r] = S[inv[r]] or zeros, for every dense row r (COPY); or (!COPY) zeros
// for the rows with inv[r] < 0 only, the others untouched and S unused.  One
// block of ty rows each, dispatched in row order, so the chip writes one
// moving window of the output.
template <bool COPY>
__global__ __launch_bounds__(kThreads) void scatter_fill_kernel(const i32x4* __restrict__ S,
                                                                const int32_t* __restrict__ inv,
                                                                int64_t n_dense, int64_t n_rows,
                                                                int vpr, i32x4* __restrict__ D) {
  const int64_t r = (int64_t)blockIdx.x * blockDim.y + threadIdx.y;
  if (r >= n_dense) return;
  const int32_t s = inv[r];
  if (!COPY && s >= 0) return;
  const bool ok = COPY && s >= 0 && s < n_rows;
  const i32x4* src = S + (int64_t)s * vpr;
  i32x4* dst = D + r * vpr;
  for (int q = threadIdx.x; q < vpr; q += blockDim.x) {
    i32x4 val = {0, 0, 0, 0};
    if (ok) val = src[q];
    __builtin_nontemporal_store(val, dst + q);
  }
}

// D holding the zero-fill scatter of the previous active set (prev) updated
// to this set's: threads t < prev_rows zero the rows of the previous set that
// are inactive now, the others write this set's rows.  The two parts touch
// different rows (a row is zeroed only when inactive now), so one launch
// does both in any order.
__global__ __launch_bounds__(kThreads) void scatter_update_kernel(
    const i32x4* __restrict__ S, const int32_t* __restrict__ inv, const int2* __restrict__ coords,
    int64_t n_rows, const int2* __restrict__ prev, int64_t prev_rows, int32_t B, int32_t V,
    int vpr, i32x4* __restrict__ D) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.y + threadIdx.y;
  if (t >= prev_rows + n_rows) return;
  const bool clear = t < prev_rows;
  const int64_t i = t - prev_rows;  // this set's row (when !clear)
  const int2 c = clear ? prev[t] : coords[i];
  if (!(c.x >= 0 && c.x < B && c.y >= 0 && c.y < V)) return;
  const int64_t r = (int64_t)c.x * V + c.y;
  if (clear && inv[r] >= 0) return;
  i32x4* dst = D + r * vpr;
  for (int q = threadIdx.x; q < vpr; q += blockDim.x) {
    i32x4 val = {0, 0, 0, 0};
    if (!clear) val = S[i * vpr + q];
    __builtin_nontemporal_store(val, dst + q);
  }
}

// D[b_i * V + v_i] = S[i] for every active row i; other rows untouched.
__global__ __launch_bounds__(kThreads) void scatter_active_kernel(const i32x4* __restrict__ S,
                                                                  const int2* __restrict__ coords,
                                                                  int64_t n_rows, int32_t B,
                                                                  int32_t V, int vpr,
                                                                  i32x4* __restrict__ D) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.y + threadIdx.y;
  if (i >= n_rows) return;
  const int2 c = coords[i];
  if (!(c.x >= 0 && c.x < B && c.y >= 0 && c.y < V)) return;
  const i32x4* src = S + i * vpr;
  i32x4* dst = D + ((int64_t)c.x * V + c.y) * vpr;
  for (int q = threadIdx.x; q < vpr; q += blockDim.x) dst[q] = src[q];
}

// ---------------------------------------------------------------------------
// segmented max-pool: one block per body.  Each thread keeps the running
// maximum of one 16-byte vector of channels over rows lo + ty_id, lo + ty_id + ty, ...
// (values widened to fp32, which is exact for bf16), then the ty partial
// maxima are combined through LDS.  NaN is the "no value yet" state:
// fmaxf(NaN, a) = a, so NaNs in the data lose to numbers as maxNum requires.
// ---------------------------------------------------------------------------

template <bool BF16>
struct PoolVec;

template <>
struct PoolVec<false> {  // 4 fp32 channels
  static constexpr int N = 4;
  __device__ static void widen(const i32x4& v, float* f) {
    for (int k = 0; k < 4; ++k) f[k] = __int_as_float(v[k]);
  }
  __device__ static i32x4 narrow(const float* f) {
    return i32x4{__float_as_int(f[0]), __float_as_int(f[1]), __float_as_int(f[2]),
                 __float_as_int(f[3])};
  }
};

template <>
struct PoolVec<true> {  // 8 bf16 channels
  static constexpr int N = 8;
  __device__ static void widen(const i32x4& v, float* f) {
    for (int k = 0; k < 4; ++k) {
      const uint32_t u = (uint32_t)v[k];
      f[2 * k] = bf16_bits_to_f32(u & 0xFFFFu);
      f[2 * k + 1] = bf16_bits_to_f32(u >> 16);
    }
  }
  __device__ static i32x4 narrow(const float* f) {
    i32x4 r;
    for (int k = 0; k < 4; ++k)
      r[k] = (int)(f32_to_bf16_bits(f[2 * k]) | (f32_to_bf16_bits(f[2 * k + 1]) << 16));
    return r;
  }
};

// Blocks (segment b, channel part): a part is a run of vpp of the row's vpr
// 16-byte vectors (all of them when there is one part); tx threads span it,
// ty row slots; each thread folds kPoolRows rows per batch, all loaded before
// the first maximum.  A row index past the segment clamps to its last row:
// repeating a row leaves a maximum unchanged, so no select is needed.  The
// parts split few, long segments over more CUs; each part's maximum is its
// own, so no block combines another's.
constexpr int kPoolThreads = 1024;
constexpr int kPoolRows = 8;
constexpr int kPoolMinBlocks = 512;   // split channels until about this many blocks
constexpr int kPoolMinPartVecs = 4;   // ... keeping at least 64 bytes of a row per part

template <bool BF16>
__global__ __launch_bounds__(kPoolThreads) void segment_max_kernel(
    const i32x4* __restrict__ S, const int32_t* __restrict__ row_ptr, int64_t n_rows, int vpr,
    int vpp, float empty_value, i32x4* __restrict__ P) {
  using PV = PoolVec<BF16>;
  extern __shared__ float part[];  // [ty][tx][N]
  const int b = blockIdx.x;
  const int qp = blockIdx.y * vpp;  // first vector of this block's channel part
  int64_t lo = row_ptr[b], hi = row_ptr[b + 1];
  lo = lo < 0 ? 0 : (lo > n_rows ? n_rows : lo);
  hi = hi < lo ? lo : (hi > n_rows ? n_rows : hi);
  const int tx = blockDim.x, ty = blockDim.y, y = threadIdx.y;
  const float nanv = __builtin_nanf("");
  for (int q0 = 0; q0 < vpp; q0 += tx) {
    const int q = qp + min(q0 + (int)threadIdx.x, vpp - 1);
    float m[PV::N];
    for (int k = 0; k < PV::N; ++k) m[k] = nanv;
    for (int64_t i0 = lo + y; i0 < hi; i0 += (int64_t)kPoolRows * ty) {
      i32x4 v[kPoolRows];
#pragma unroll
      for (int r = 0; r < kPoolRows; ++r) v[r] = S[min(i0 + (int64_t)r * ty, hi - 1) * vpr + q];
#pragma unroll
      for (int r = 0; r < kPoolRows; ++r) {
        float f[PV::N];
        PV::widen(v[r], f);
        for (int k = 0; k < PV::N; ++k) m[k] = fmaxf(m[k], f[k]);
      }
    }
    // fold the ty partial maxima: slots y >= 8 into y % 8, then 1..7 into 0
    float* mine = part + ((size_t)y * tx + threadIdx.x) * PV::N;
    for (int k = 0; k < PV::N; ++k) mine[k] = m[k];
    __syncthreads();
    if (y < 8) {
      for (int yy = y + 8; yy < ty; yy += 8) {
        const float* o = part + ((size_t)yy * tx + threadIdx.x) * PV::N;
        for (int k = 0; k < PV::N; ++k) m[k] = fmaxf(m[k], o[k]);
      }
      for (int k = 0; k < PV::N; ++k) mine[k] = m[k];
    }
    __syncthreads();
    if (y == 0 && q0 + (int)threadIdx.x < vpp) {
      for (int yy = 1; yy < 8 && yy < ty; ++yy) {
        const float* o = part + ((size_t)yy * tx + threadIdx.x) * PV::N;
        for (int k = 0; k < PV::N; ++k) m[k] = fmaxf(m[k], o[k]);
      }
      if (hi == lo)
        for (int k = 0; k < PV::N; ++k) m[k] = empty_value;
      P[(int64_t)b * vpr + q] = PV::narrow(m);
    }
    __syncthreads();
  }
}

}  // namespace

hipError_t launch_gather(const void* x, const int32_t* coords, int64_t n_rows, int32_t B,
                         int32_t V, int32_t row_bytes, void* S, hipStream_t stream) {
  return launch_gather_ext(x, nullptr, 0, coords, n_rows, B, B, V, row_bytes, S, stream);
}

hipError_t launch_gather_ext(const void* x, const uint8_t* me, int mask_mode,
                             const int32_t* coords, int64_t n_rows, int32_t B, int32_t Bx,
                             int32_t V, int32_t row_bytes, void* S, hipStream_t stream) {
  if (n_rows <= 0) return hipSuccess;
  const RowShape s = row_shape(row_bytes);
  const int64_t per_block = (int64_t)s.ty * kGatherRows;
  const int64_t blocks = (n_rows + per_block - 1) / per_block;
  const auto* xv = static_cast<const i32x4*>(x);
  const auto* cv = reinterpret_cast<const int2*>(coords);
  auto* sv = static_cast<i32x4*>(S);
  if (mask_mode == 1)
    hipLaunchKernelGGL(gather_kernel<1>, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0, stream, xv,
                       me, cv, n_rows, B, Bx, V, s.vpr, sv);
  else if (mask_mode == 2)
    hipLaunchKernelGGL(gather_kernel<2>, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0, stream, xv,
                       me, cv, n_rows, B, Bx, V, s.vpr, sv);
  else
    hipLaunchKernelGGL(gather_kernel<0>, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0, stream, xv,
                       me, cv, n_rows, B, Bx, V, s.vpr, sv);
  return hipGetLastError();
}

hipError_t launch_combine(const void* Y, int32_t kappa, int64_t rows, int32_t row_bytes, int op,
                          int is_bf16, void* out, hipStream_t stream) {
  const int64_t n_vec = rows * (row_bytes / 16);
  if (n_vec <= 0) return hipSuccess;
  const int64_t blocks = (n_vec + kThreads - 1) / kThreads;
  const auto* y = static_cast<const i32x4*>(Y);
  auto* o = static_cast<i32x4*>(out);
#define SHC_COMBINE(OPV, BF)                                                                \
  if (op == OPV && (is_bf16 != 0) == BF)                                                    \
    hipLaunchKernelGGL((combine_kernel<OPV, BF>), dim3((unsigned)blocks), dim3(kThreads), 0, \
                       stream, y, kappa, n_vec, o);
  SHC_COMBINE(0, true) SHC_COMBINE(1, true) SHC_COMBINE(2, true)
  SHC_COMBINE(0, false) SHC_COMBINE(1, false) SHC_COMBINE(2, false)
#undef SHC_COMBINE
  return hipGetLastError();
}

hipError_t launch_row_activity(const uint8_t* me, int32_t B, int32_t V, int32_t C, uint8_t* m,
                               hipStream_t stream) {
  const int64_t n_vert = (int64_t)B * V;
  const int vpr = C / 16;  // 16-byte chunks of mask bytes per vertex
  int tx = 1;              // lanes per vertex: a power of two <= min(vpr, 64)
  while (2 * tx <= vpr && 2 * tx <= 64) tx *= 2;
  const int64_t threads = n_vert * tx;
  const int64_t blocks = (threads + kThreads - 1) / kThreads;
  hipLaunchKernelGGL(row_activity_kernel, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                     reinterpret_cast<const i32x4*>(me), n_vert, vpr, tx, m);
  return hipGetLastError();
}

hipError_t launch_scatter(const void* S, const int32_t* inv, const int32_t* coords,
                          int64_t n_rows, int32_t B, int32_t V, int32_t row_bytes, int zero_fill,
                          void* D, hipStream_t stream) {
  const RowShape s = row_shape(row_bytes);
  if (zero_fill) {
    const int64_t n_dense = (int64_t)B * V;
    const int64_t blocks = (n_dense + s.ty - 1) / s.ty;
    hipLaunchKernelGGL(scatter_fill_kernel<true>, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0,
                       stream, static_cast<const i32x4*>(S), inv, n_dense, n_rows, s.vpr,
                       static_cast<i32x4*>(D));
  } else {
    if (n_rows == 0) return hipSuccess;
    const int64_t blocks = (n_rows + s.ty - 1) / s.ty;
    hipLaunchKernelGGL(scatter_active_kernel, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0,
                       stream, static_cast<const i32x4*>(S),
                       reinterpret_cast<const int2*>(coords), n_rows, B, V, s.vpr,
                       static_cast<i32x4*>(D));
  }
  return hipGetLastError();
}

hipError_t launch_scatter_update(const void* S, const int32_t* inv, const int32_t* coords,
                                 int64_t n_rows, const int32_t* prev_coords, int64_t prev_rows,
                                 int32_t B, int32_t V, int32_t row_bytes, void* D,
                                 hipStream_t stream) {
  const RowShape s = row_shape(row_bytes);
  const int64_t rows = prev_rows + n_rows;
  if (rows == 0) return hipSuccess;
  const int64_t blocks = (rows + s.ty - 1) / s.ty;
  hipLaunchKernelGGL(scatter_update_kernel, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0, stream,
                     static_cast<const i32x4*>(S), inv, reinterpret_cast<const int2*>(coords),
                     n_rows, reinterpret_cast<const int2*>(prev_coords), prev_rows, B, V, s.vpr,
                     static_cast<i32x4*>(D));
  return hipGetLastError();
}

hipError_t launch_clear_inactive(const int32_t* inv, int32_t B, int32_t V, int32_t row_bytes,
                                 void* D, hipStream_t stream) {
  const RowShape s = row_shape(row_bytes);
  const int64_t n_dense = (int64_t)B * V;
  const int64_t blocks = (n_dense + s.ty - 1) / s.ty;
  hipLaunchKernelGGL(scatter_fill_kernel<false>, dim3((unsigned)blocks), dim3(s.tx, s.ty), 0,
                     stream, nullptr, inv, n_dense, (int64_t)0, s.vpr, static_cast<i32x4*>(D));
  return hipGetLastError();
}

hipError_t launch_segment_max(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                              int32_t C, int is_bf16, float empty_value, void* P,
                              hipStream_t stream) {
  const int32_t row_bytes = C * (is_bf16 ? 2 : 4);
  const int vpr = row_bytes / 16;
  int parts = 1;
  while ((int64_t)B * parts < kPoolMinBlocks && vpr % (2 * parts) == 0 &&
         vpr / (2 * parts) >= kPoolMinPartVecs)
    parts *= 2;
  const int vpp = vpr / parts;
  RowShape s = row_shape(vpp * 16);
  // a split segment's rows are spread over 4x fewer threads per block
  s.ty = (parts > 1 ? kPoolThreads / 4 : kPoolThreads) / s.tx;
  if (s.ty < 1) s.ty = 1;
  const int n_per_vec = is_bf16 ? 8 : 4;
  const size_t lds = (size_t)s.tx * s.ty * n_per_vec * sizeof(float);
  if (is_bf16)
    hipLaunchKernelGGL(segment_max_kernel<true>, dim3(B, parts), dim3(s.tx, s.ty), lds, stream,
                       static_cast<const i32x4*>(S), row_ptr, n_rows, vpr, vpp, empty_value,
                       static_cast<i32x4*>(P));
  else
    hipLaunchKernelGGL(segment_max_kernel<false>, dim3(B, parts), dim3(s.tx, s.ty), lds, stream,
                       static_cast<const i32x4*>(S), row_ptr, n_rows, vpr, vpp, empty_value,
                       static_cast<i32x4*>(P));
  return hipGetLastError();
}

}  // namespace shc
