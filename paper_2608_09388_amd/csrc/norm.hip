// Sparse group normalization (Eqs. 7-9): for every body b (a segment of the
// active rows, [row_ptr[b], row_ptr[b+1])) and every group g of C/G
// consecutive channels,
//
//   mu  = mean of the group's values over the body's rows          (Eq. 7)
//   var = mean of (value - mu)^2 over the same values              (Eq. 8)
//   out = (value - mu) / sqrt(var + eps)                           (Eq. 9)
//
// Only active rows enter the statistics (the rows of S are the active ones).
//
// Workgroups of 1024 threads, F per body: workgroup (b, f) takes the f-th
// of F equal channel ranges (whole groups), so B * F workgroups fill the
// chip even when bodies are few.  Thread (tx, ty) owns 16-byte channel
// vector tx of its range in rows ty, ty + TY, ...; its partial sums are per
// channel (4 fp32 or 8 bf16 channels), summed over the rows a wavefront holds
// with lane shuffles, then through LDS over the wavefronts, then over the
// channels of each group.  The statistics are
// two-pass: the mean, held in fp64 from the first addition on, then the
// squared deviations from it, summed in fp32 over a thread's rows (at most 16
// positive terms) and in fp64 from there; the variance errs by at most about
// 16 * 2^-24 relative and the mean by n * 2^-53 of the values' magnitude.  Every
// output is ((value - mu_hi) - mu_lo) * rs in fp32, with the fp64 mean split
// into two fp32 terms and rs = 1/sqrt(var + eps) rounded to fp32: four
// roundings of about 2^-24 of the output each (then bf16's for bf16 outputs).
// The in-wavefront row sums use DPP rotations and the row/half swaps of
// v_permlane16_swap / v_permlane32_swap (VALU, no LDS traffic).
// A body of up to kResident vectors per thread stays in registers, so HBM
// sees one read and one write of every value; a larger body is streamed
// three times (sums, deviations, output), the later passes mostly from L2.
#include <algorithm>
#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kNormThreads = 1024;
constexpr int kResident = 16;  // vectors per thread held in registers

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

template <bool BF16>
struct NormVec;
template <>
struct NormVec<false> {
  static constexpr int N = 4;
  static __device__ __forceinline__ void widen(const i32x4& v, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = __int_as_float(v[e]);
  }
  static __device__ __forceinline__ i32x4 narrow(const float* f) {
    return i32x4{__float_as_int(f[0]), __float_as_int(f[1]), __float_as_int(f[2]),
                 __float_as_int(f[3])};
  }
};
template <>
struct NormVec<true> {
  static constexpr int N = 8;
  static __device__ __forceinline__ void widen(const i32x4& v, float* f) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {  // bf16 -> fp32 is exact: the bits move up
      f[2 * e] = __int_as_float(v[e] << 16);
      f[2 * e + 1] = __int_as_float(v[e] & (int)0xFFFF0000);
    }
  }
  static __device__ __forceinline__ i32x4 narrow(const float* f) {
    i32x4 out;
#pragma unroll
    for (int e = 0; e < 4; ++e) {  // hardware round-to-nearest-even conversion
      const bf16x2 h = __builtin_convertvector(f32x2{f[2 * e], f[2 * e + 1]}, bf16x2);
      out[e] = __builtin_bit_cast(int, h);
    }
    return out;
  }
};

// Sum of v over the lanes of a wavefront that share lane % tx (tx a power of
// two below 64): rotations within each 16-lane row (DPP), then the swaps of
// rows 16 apart and halves 32 apart (v_permlane16_swap / v_permlane32_swap).
// All VALU; every lane ends with its sum.
__device__ __forceinline__ double rot_row(double v, int d) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  int lo = (int)(uint32_t)u, hi = (int)(uint32_t)(u >> 32);
  switch (d) {
    case 1: lo = __builtin_amdgcn_update_dpp(0, lo, 0x121, 0xF, 0xF, false);
            hi = __builtin_amdgcn_update_dpp(0, hi, 0x121, 0xF, 0xF, false); break;
    case 2: lo = __builtin_amdgcn_update_dpp(0, lo, 0x122, 0xF, 0xF, false);
            hi = __builtin_amdgcn_update_dpp(0, hi, 0x122, 0xF, 0xF, false); break;
    case 4: lo = __builtin_amdgcn_update_dpp(0, lo, 0x124, 0xF, 0xF, false);
            hi = __builtin_amdgcn_update_dpp(0, hi, 0x124, 0xF, 0xF, false); break;
    default: lo = __builtin_amdgcn_update_dpp(0, lo, 0x128, 0xF, 0xF, false);
             hi = __builtin_amdgcn_update_dpp(0, hi, 0x128, 0xF, 0xF, false); break;
  }
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
__device__ __forceinline__ double lanes_sum(double v, int tx) {
  for (int d = tx; d < 16; d <<= 1) v += rot_row(v, d);
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)u, hi = (uint32_t)(u >> 32);
  if (tx <= 16) {
    const auto a = __builtin_amdgcn_permlane16_swap(lo, lo, false, false);
    const auto b = __builtin_amdgcn_permlane16_swap(hi, hi, false, false);
    v = __builtin_bit_cast(double, ((uint64_t)b[0] << 32) | a[0]) +
        __builtin_bit_cast(double, ((uint64_t)b[1] << 32) | a[1]);
  }
  const uint64_t w = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo2 = (uint32_t)w, hi2 = (uint32_t)(w >> 32);
  const auto c = __builtin_amdgcn_permlane32_swap(lo2, lo2, false, false);
  const auto d2 = __builtin_amdgcn_permlane32_swap(hi2, hi2, false, false);
  return __builtin_bit_cast(double, ((uint64_t)d2[0] << 32) | c[0]) +
         __builtin_bit_cast(double, ((uint64_t)d2[1] << 32) | c[1]);
}

template <bool BF16>
__global__ __launch_bounds__(kNormThreads) void group_norm_kernel(
    const i32x4* __restrict__ S, const int32_t* __restrict__ row_ptr, int64_t n_rows, int C,
    int G, float eps, int vpr, i32x4* __restrict__ out) {
  using NV = NormVec<BF16>;
  constexpr int N = NV::N;
  // part[slot][Cl]: channel partials (one slot per thread row, or per
  // wavefront after the shuffles); then chan[Cl]; then stat[Cl], the group's
  // mean / reciprocal deviation broadcast back per channel, which reuses the
  // partials' space (every read of part precedes a barrier before stat is
  // written, and a barrier at the start of each reduction keeps the next
  // partials from overwriting stat while it is still being read)
  extern __shared__ double smem[];
  const int TX = blockDim.x, TY = blockDim.y;  // TX = vectors of this workgroup's range
  const int ty = threadIdx.y;
  const int tid = ty * TX + threadIdx.x;
  const int Cl = TX * N;                       // channels of the range
  const int tx = blockIdx.y * TX + threadIdx.x;  // vector within the row
  // rows a wavefront holds: 64 / TX when TX divides 64 (then reduced by shuffles)
  const int rw = (TX <= 64 && 64 % TX == 0) ? 64 / TX : 1;
  const int slots = rw > 1 ? (TX * TY) / 64 : TY;
  double* part = smem;                // [slots][Cl]
  double* chan = smem + slots * Cl;   // [Cl]
  double* stat = smem;                // [Cl]: the group's mean, then 1/sqrt(var + eps)

  int64_t lo = row_ptr[blockIdx.x], hi = row_ptr[blockIdx.x + 1];
  lo = lo < 0 ? 0 : (lo > n_rows ? n_rows : lo);
  hi = hi < lo ? lo : (hi > n_rows ? n_rows : hi);
  const int rows = (int)(hi - lo);
  if (rows == 0) return;  // uniform over the workgroup
  const bool resident = rows <= TY * kResident;
  const int cg = C / G;
  const double count = (double)rows * (double)cg;  // exact
  const double deps = (double)eps;

  // this thread's channel partials -> per-channel totals over the rows ->
  // per group, into stat[] (the range's channels hold whole groups)
  auto reduce = [&](double* acc, bool second) {
    __syncthreads();  // the previous reduction's stat has been read
    if (rw > 1) {
      const int lane = tid & 63;
#pragma unroll
      for (int e = 0; e < N; ++e) acc[e] = lanes_sum(acc[e], TX);
      if (lane < TX)
#pragma unroll
        for (int e = 0; e < N; ++e) part[(tid >> 6) * Cl + threadIdx.x * N + e] = acc[e];
    } else {
#pragma unroll
      for (int e = 0; e < N; ++e) part[ty * Cl + threadIdx.x * N + e] = acc[e];
    }
    __syncthreads();
    const int nt = TX * TY;
    // groups line up with wavefront lanes: cg divides 64, or 64 divides cg
    if (Cl <= nt && ((cg <= 64 && 64 % cg == 0) || cg % 64 == 0)) {
      // thread c: channel total (four independent partial sums), then the
      // group total by lane shuffles (cg <= 64) or per-wave partials (cg > 64)
      const int c = tid;
      double t = 0.0;
      if (c < Cl) {
        double q[4] = {0.0, 0.0, 0.0, 0.0};
        int y = 0;
        for (; y + 4 <= slots; y += 4)
#pragma unroll
          for (int u = 0; u < 4; ++u) q[u] += part[(y + u) * Cl + c];
        for (; y < slots; ++y) q[0] += part[y * Cl + c];
        t = (q[0] + q[1]) + (q[2] + q[3]);
      }
      const int span = cg < 64 ? cg : 64;  // lanes summed by shuffles
      for (int d = 1; d < span; d <<= 1) t += __shfl_xor(t, d, 64);
      if (cg <= 64) {
        if (c < Cl && c % cg == 0) {
          const double v = t / count;  // correctly rounded: an exact mean stays exact
          chan[c] = second ? 1.0 / sqrt(v + deps) : v;  // the group's first channel
        }
      } else if (c < Cl && (c & 63) == 0) {
        chan[c] = t;  // wave partial of the group, at the wave's first channel
      }
      __syncthreads();
      if (cg > 64) {
        for (int g = tid; g < Cl / cg; g += nt) {
          double u = 0.0;
          for (int w = g * cg; w < (g + 1) * cg; w += 64) u += chan[w];
          const double v = u / count;
          chan[g * cg] = second ? 1.0 / sqrt(v + deps) : v;
        }
        __syncthreads();
      }
    } else {
      for (int c = tid; c < Cl; c += nt) {
        double t = 0.0;
        for (int y = 0; y < slots; ++y) t += part[y * Cl + c];
        chan[c] = t;
      }
      __syncthreads();
      for (int g = tid; g < Cl / cg; g += nt) {
        double t = 0.0;
        for (int c = g * cg; c < (g + 1) * cg; ++c) t += chan[c];
        const double v = t / count;  // correctly rounded: an exact mean stays exact
        chan[g * cg] = second ? 1.0 / sqrt(v + deps) : v;  // the group's first channel
      }
      __syncthreads();
    }
    for (int c = tid; c < Cl; c += nt) stat[c] = chan[(c / cg) * cg];
    __syncthreads();
  };

  i32x4 keep[kResident];
  double acc[N];
  // ---- pass 1: sums ------------------------------------------------------------
#pragma unroll
  for (int e = 0; e < N; ++e) acc[e] = 0.0;
  if (resident) {
#pragma unroll
    for (int k = 0; k < kResident; ++k) {
      const int r = ty + k * TY;
      keep[k] = i32x4{0, 0, 0, 0};
      if (k * TY < rows && r < rows) keep[k] = S[(lo + r) * vpr + tx];
    }
#pragma unroll
    for (int k = 0; k < kResident; ++k) {
      if (k * TY < rows) {  // uniform: register slots no thread of the body uses are skipped
        float f[N];
        NV::widen(keep[k], f);  // zeros past the rows add nothing
#pragma unroll
        for (int e = 0; e < N; ++e) acc[e] += (double)f[e];
      }
    }
  } else {
    for (int r = ty; r < rows; r += TY) {
      float f[N];
      NV::widen(S[(lo + r) * vpr + tx], f);
#pragma unroll
      for (int e = 0; e < N; ++e) acc[e] += (double)f[e];
    }
  }
  reduce(acc, false);
  double mu[N];
#pragma unroll
  for (int e = 0; e < N; ++e) mu[e] = stat[threadIdx.x * N + e];
  // the mean as two fp32 terms (hi + lo): centred values (value - mu_hi) - mu_lo
  // err by 2^-24 of themselves, not of the mean
  float mu_hi[N], mu_lo[N];
#pragma unroll
  for (int e = 0; e < N; ++e) {
    mu_hi[e] = (float)mu[e];
    mu_lo[e] = (float)(mu[e] - (double)mu_hi[e]);
  }

  // ---- pass 2: squared deviations from the group mean --------------------------
  // A thread's squares (positive terms) are summed in fp32 over at most
  // kResident rows at a time (relative error at most 15 * 2^-24), then the
  // sums go on in fp64.
#pragma unroll
  for (int e = 0; e < N; ++e) acc[e] = 0.0;
  if (resident) {
    float sq[N];
#pragma unroll
    for (int e = 0; e < N; ++e) sq[e] = 0.f;
#pragma unroll
    for (int k = 0; k < kResident; ++k) {
      if (k * TY < rows) {  // uniform skip, then the rows of this slot
        const bool in = ty + k * TY < rows;
        float f[N];
        NV::widen(keep[k], f);
#pragma unroll
        for (int e = 0; e < N; ++e) {
          const float d = in ? (f[e] - mu_hi[e]) - mu_lo[e] : 0.f;
          sq[e] = __builtin_fmaf(d, d, sq[e]);
        }
      }
    }
#pragma unroll
    for (int e = 0; e < N; ++e) acc[e] = (double)sq[e];
  } else {
    for (int r0 = ty; r0 < rows; r0 += kResident * TY) {
      float sq[N];
#pragma unroll
      for (int e = 0; e < N; ++e) sq[e] = 0.f;
      for (int r = r0; r < rows && r < r0 + kResident * TY; r += TY) {
        float f[N];
        NV::widen(S[(lo + r) * vpr + tx], f);
#pragma unroll
        for (int e = 0; e < N; ++e) {
          const float d = (f[e] - mu_hi[e]) - mu_lo[e];
          sq[e] = __builtin_fmaf(d, d, sq[e]);
        }
      }
#pragma unroll
      for (int e = 0; e < N; ++e) acc[e] += (double)sq[e];
    }
  }
  reduce(acc, true);
  double rs[N];
#pragma unroll
  for (int e = 0; e < N; ++e) rs[e] = stat[threadIdx.x * N + e];

  // ---- pass 3: normalized values -----------------------------------------------
  float rs_f[N];
#pragma unroll
  for (int e = 0; e < N; ++e) rs_f[e] = (float)rs[e];
  auto emit = [&](const i32x4& v, int r) {
    float f[N];
    NV::widen(v, f);
#pragma unroll
    for (int e = 0; e < N; ++e) f[e] = ((f[e] - mu_hi[e]) - mu_lo[e]) * rs_f[e];
    __builtin_nontemporal_store(NV::narrow(f), out + (lo + r) * vpr + tx);
  };
  if (resident) {
#pragma unroll
    for (int k = 0; k < kResident; ++k)
      if (k * TY < rows && ty + k * TY < rows) emit(keep[k], ty + k * TY);
  } else {
    for (int r = ty; r < rows; r += TY) emit(S[(lo + r) * vpr + tx], r);
  }
}

}  // namespace

// Channel ranges per body: the largest power of two F <= num_cus / B (one
// 1024-thread workgroup fits a CU, so one wave of workgroups) that
// splits the row's vectors evenly, keeps whole groups in every range and
// leaves every workgroup at least 64 contiguous bytes of each row.
int group_norm_split(int32_t B, int32_t C, int32_t G, int is_bf16, int num_cus) {
  const int vpr = C * (is_bf16 ? 2 : 4) / 16;
  const int cg = C / G;
  const int want = std::max(1, num_cus / std::max(1, (int)B));
  int f = 1;
  while (2 * f <= want && vpr % (2 * f) == 0 && vpr / (2 * f) >= 4 && (C / (2 * f)) % cg == 0)
    f *= 2;
  return f;
}

size_t group_norm_lds_bytes(int32_t C, int is_bf16, int split) {
  const int tx = C * (is_bf16 ? 2 : 4) / 16 / split;
  const int ty = kNormThreads / tx;
  const int cl = C / split;
  // partials (at most ty slots in either layout; stat reuses them) + chan
  return (size_t)(ty + 1) * (size_t)cl * sizeof(double);
}

hipError_t launch_group_norm(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                             int32_t C, int32_t G, float eps, int is_bf16, void* out,
                             int num_cus, hipStream_t stream) {
  const int vpr = C * (is_bf16 ? 2 : 4) / 16;  // <= 1024 for C <= 4096
  const int split = group_norm_split(B, C, G, is_bf16, num_cus);
  const dim3 block(vpr / split, kNormThreads / (vpr / split));
  const size_t lds = group_norm_lds_bytes(C, is_bf16, split);
  // up to 96 KB of dynamic LDS (C = 4096 bf16): allow it once per instantiation
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [&] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(group_norm_kernel<true>),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
    if (attr_err == hipSuccess)
      attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(group_norm_kernel<false>),
                                     hipFuncAttributeMaxDynamicSharedMemorySize, 96 * 1024);
  });
  if (attr_err != hipSuccess) return attr_err;
  if (B <= 0 || n_rows <= 0) return hipSuccess;
  if (is_bf16)
    hipLaunchKernelGGL(group_norm_kernel<true>, dim3(B, split), block, lds, stream,
                       static_cast<const i32x4*>(S), row_ptr, n_rows, C, G, eps, vpr,
                       static_cast<i32x4*>(out));
  else
    hipLaunchKernelGGL(group_norm_kernel<false>, dim3(B, split), block, lds, stream,
                       static_cast<const i32x4*>(S), row_ptr, n_rows, C, G, eps, vpr,
                       static_cast<i32x4*>(out));
  return hipGetLastError();
}

}  // namespace shc
