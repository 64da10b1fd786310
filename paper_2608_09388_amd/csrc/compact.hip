// Mask compaction: the decomposition of Eq. 2 (coordinate list C' of the
// active (b, v) entries, in (b, v) order), plus the inverse map, the per-body
// row offsets and the active count.
//
// Two launches over the flattened mask of B*V bytes:
//   1. count   -- every block counts the non-zero bytes of its span;
//   2. write   -- every block sums the counts of the blocks before it (block
//                 0 sums them all and publishes N' -- row_ptr[B], the device
//                 and the host count -- before writing anything else, so a
//                 host waiting for the count wakes while the lists are still
//                 being written), then walks its span in chunks of 4096 entries.  Inside a chunk a
//                 thread owns four 4-byte groups (one per 1024-entry
//                 sub-chunk, so each load and each int4 store of `inv` is
//                 contiguous across the wavefront); the four per-thread counts
//                 are packed in 16-bit fields and scanned together with one
//                 wavefront shuffle scan and one LDS pass over the 4 waves.
// Integer work only: the result is the same on every run.
#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kChunk = kThreads * 4 * 4;  // entries per chunk
constexpr int kSub = kThreads * 4;        // entries per sub-chunk

// 0x80 in every byte of `w` that is non-zero, 0 elsewhere.
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t w) {
  return (((w & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | w) & 0x80808080u;
}

__device__ __forceinline__ uint32_t wave_inclusive_scan(uint32_t x) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

// Block-wide sum; every thread gets the total.
__device__ __forceinline__ uint32_t block_sum(uint32_t x, uint32_t* red) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, 64);
  const int wave = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[wave] = x;
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) t += red[w];
  return t;
}

// Four 4-byte groups of the chunk starting at `c0` owned by this thread; bytes
// at or past `end` read as zero.
__device__ __forceinline__ void load_groups(const uint8_t* mask, int64_t c0, int64_t end,
                                            uint32_t w[4]) {
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const int64_t e = c0 + (int64_t)k * kSub + (int64_t)threadIdx.x * 4;
    if (e + 4 <= end) {
      w[k] = *reinterpret_cast<const uint32_t*>(mask + e);
    } else {
      uint32_t v = 0;
      for (int q = 0; q < 4; ++q)
        if (e + q < end) v |= (uint32_t)mask[e + q] << (8 * q);
      w[k] = v;
    }
  }
}

__global__ __launch_bounds__(kThreads) void compact_count_kernel(const uint8_t* __restrict__ mask,
                                                                 int64_t total, int64_t per_block,
                                                                 int32_t* __restrict__ counts) {
  __shared__ uint32_t red[kWaves];
  const int64_t start = (int64_t)blockIdx.x * per_block;
  const int64_t end = min(start + per_block, total);
  uint32_t cnt = 0;
  for (int64_t c0 = start; c0 < end; c0 += kChunk) {
    uint32_t w[4];
    load_groups(mask, c0, end, w);
#pragma unroll
    for (int k = 0; k < 4; ++k) cnt += __popc(nonzero_bytes(w[k]));
  }
  cnt = block_sum(cnt, red);
  if (threadIdx.x == 0) counts[blockIdx.x] = (int32_t)cnt;
}

__global__ __launch_bounds__(kThreads) void compact_write_kernel(
    const uint8_t* __restrict__ mask, int64_t total, int64_t per_block, int32_t B, int32_t V,
    const int32_t* __restrict__ counts, int32_t* __restrict__ coords, int32_t* __restrict__ inv,
    int32_t* __restrict__ row_ptr, int32_t* __restrict__ n_active, int64_t* n_host, int64_t cap) {
  __shared__ uint32_t red[kWaves];
  __shared__ uint32_t wave_tot[2][kWaves];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;

  const int64_t start = (int64_t)blockIdx.x * per_block;
  const int64_t end = min(start + per_block, total);
  // the first chunk's mask bytes are loaded while the prefix below is formed
  uint32_t w[4];
  load_groups(mask, start, end, w);

  // rows taken by the blocks before this one (block 0: by every block, N')
  const int upto = blockIdx.x == 0 ? (int)gridDim.x : (int)blockIdx.x;
  uint32_t before = 0;
  for (int q = tid; q < upto; q += kThreads) before += (uint32_t)counts[q];
  int64_t base = block_sum(before, red);
  if (blockIdx.x == 0) {
    if (tid == 0) {
      row_ptr[B] = (int32_t)base;
      *n_active = (int32_t)base;
      // page-locked host copy of the count: a system-scope store
      if (n_host != nullptr) __hip_atomic_store(n_host, base, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    base = 0;
  }

  for (int64_t c0 = start; c0 < end; c0 += kChunk) {
    uint32_t nz[4];
    if (c0 != start) load_groups(mask, c0, end, w);
    // per-thread counts of the four groups, packed 16 bits each (a block sum
    // per field is at most 1024, so the fields never carry into each other)
    uint32_t lo = 0, hi = 0;
#pragma unroll
    for (int k = 0; k < 4; ++k) nz[k] = nonzero_bytes(w[k]);
    lo = (uint32_t)__popc(nz[0]) | ((uint32_t)__popc(nz[1]) << 16);
    hi = (uint32_t)__popc(nz[2]) | ((uint32_t)__popc(nz[3]) << 16);
    const uint32_t lo_inc = wave_inclusive_scan(lo);
    const uint32_t hi_inc = wave_inclusive_scan(hi);
    __syncthreads();  // wave_tot reuse across chunks
    if (lane == 63) {
      wave_tot[0][wave] = lo_inc;
      wave_tot[1][wave] = hi_inc;
    }
    __syncthreads();
    uint32_t lo_ex = lo_inc - lo, hi_ex = hi_inc - hi, lo_tot = 0, hi_tot = 0;
#pragma unroll
    for (int q = 0; q < kWaves; ++q) {
      if (q < wave) {
        lo_ex += wave_tot[0][q];
        hi_ex += wave_tot[1][q];
      }
      lo_tot += wave_tot[0][q];
      hi_tot += wave_tot[1][q];
    }
    const uint32_t tot[4] = {lo_tot & 0xFFFFu, lo_tot >> 16, hi_tot & 0xFFFFu, hi_tot >> 16};
    const uint32_t ex[4] = {lo_ex & 0xFFFFu, lo_ex >> 16, hi_ex & 0xFFFFu, hi_ex >> 16};
    int64_t sub_base = base;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int64_t e0 = c0 + (int64_t)k * kSub + (int64_t)tid * 4;
      int64_t pos = sub_base + ex[k];
      if (e0 < end) {
        int32_t b = (int32_t)(e0 / V);
        int32_t v = (int32_t)(e0 - (int64_t)b * V);
        int32_t out[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int64_t e = e0 + q;
          const bool on = (nz[k] >> (8 * q + 7)) & 1u;
          out[q] = on ? (int32_t)pos : -1;
          if (e < end) {
            if (v == 0) row_ptr[b] = (int32_t)pos;
            if (on && pos < cap) {
              coords[2 * pos] = b;
              coords[2 * pos + 1] = v;
            }
          }
          pos += on ? 1 : 0;
          if (++v == V) {
            v = 0;
            ++b;
          }
        }
        if (e0 + 4 <= end) {
          *reinterpret_cast<i32x4*>(inv + e0) = i32x4{out[0], out[1], out[2], out[3]};
        } else {
          for (int q = 0; q < 4; ++q)
            if (e0 + q < end) inv[e0 + q] = out[q];
        }
      }
      sub_base += tot[k];
    }
    base = sub_base;
  }
}

}  // namespace

void compact_plan(int64_t total, int32_t* nblocks, int64_t* per_block) {
  // at most ~1024 blocks so that the per-block prefix over earlier counts stays cheap
  int64_t span = (total + 1023) / 1024;
  span = ((span + kChunk - 1) / kChunk) * kChunk;
  if (span < kChunk) span = kChunk;
  *per_block = span;
  *nblocks = (int32_t)((total + span - 1) / span);
  if (*nblocks < 1) *nblocks = 1;
}

hipError_t launch_compact(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords, int32_t* inv,
                          int32_t* row_ptr, int32_t* n_active, int64_t* n_host, int64_t cap,
                          int32_t* block_counts, hipStream_t stream) {
  const int64_t total = (int64_t)B * V;
  int32_t nblocks;
  int64_t per_block;
  compact_plan(total, &nblocks, &per_block);
  hipLaunchKernelGGL(compact_count_kernel, dim3(nblocks), dim3(kThreads), 0, stream, mask, total,
                     per_block, block_counts);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(compact_write_kernel, dim3(nblocks), dim3(kThreads), 0, stream, mask, total,
                     per_block, B, V, block_counts, coords, inv, row_ptr, n_active, n_host, cap);
  return hipGetLastError();
}

}  // namespace shc
