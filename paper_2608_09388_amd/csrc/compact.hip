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
// A variant builds the neighbour-row table of the active set
// (neighbors.hip) in the same pass as the lists: after the count launch, one
// block per body numbers the body's rows and keeps that numbering in LDS, so
// the table entries of its rows -- whose neighbours lie in the same body --
// come from LDS rather than from a second pass over `inv`.
// Integer work only: the result is the same on every run.
#include <mutex>

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


// ---------------------------------------------------------------------------
// compaction + neighbour-row table, one block of T threads per body
// ---------------------------------------------------------------------------

// A workgroup barrier that orders LDS only: outstanding global loads and
// stores stay in flight across it (__syncthreads would wait for them all).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// LDS of the per-body numbering: padded vertex -> row map, then row -> vertex.
__host__ __device__ constexpr int compact_table_row_words(int V) { return V + V / 16 + 1; }
__host__ __device__ constexpr int compact_table_lds_bytes(int V) {
  return (compact_table_row_words(V) + V) * (int)sizeof(int32_t);
}
static_assert(compact_table_lds_bytes(kCompactTableMaxV) + 1024 <= 160 * 1024,
              "per-body numbering exceeds LDS");

// Block-wide sums of three values (every thread gets all three).
template <int T>
__device__ __forceinline__ void block_sum3(uint32_t& x, uint32_t& y, uint32_t& z,
                                           uint32_t* red) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) {
    x += __shfl_xor(x, d, 64);
    y += __shfl_xor(y, d, 64);
    z += __shfl_xor(z, d, 64);
  }
  constexpr int W = T / 64;
  const int wave = threadIdx.x >> 6;
  lds_barrier();
  if ((threadIdx.x & 63) == 0) {
    red[wave] = x;
    red[W + wave] = y;
    red[2 * W + wave] = z;
  }
  lds_barrier();
  x = y = z = 0;
#pragma unroll
  for (int w = 0; w < W; ++w) {
    x += red[w];
    y += red[W + w];
    z += red[2 * W + w];
  }
}

// third word of a raw buffer resource on gfx9-family parts (32-bit data, no swizzle)
constexpr int kBufferWord3 = 0x00020000;

// The 16-byte group g of the mask, through a buffer resource of the mask's
// bytes: a group past the end reads zeros, and the one group that reaches past
// the end is re-read byte by byte in group_flags.  No branch around the load,
// so it stays in flight until its words are used.
__device__ __forceinline__ void load_group(__amdgpu_buffer_rsrc_t rsrc, int64_t g, uint32_t w[4]) {
  const i32x4 v = __builtin_bit_cast(
      i32x4, __builtin_amdgcn_raw_buffer_load_b128(rsrc, (uint32_t)(g * 16), 0, 0));
  w[0] = (uint32_t)v[0];
  w[1] = (uint32_t)v[1];
  w[2] = (uint32_t)v[2];
  w[3] = (uint32_t)v[3];
}

// Bit q (q < 16) set when byte q of group g is non-zero.
__device__ __forceinline__ uint32_t group_flags(const uint8_t* mask, int64_t total,
                                                const uint32_t wl[4], int64_t g) {
  const int64_t e = g * 16;
  uint32_t w[4] = {wl[0], wl[1], wl[2], wl[3]};
  if (e + 16 > total) {  // the mask's last group, cut short
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      uint32_t x = 0;
      for (int q = 0; q < 4; ++q)
        if (e + 4 * k + q < total) x |= (uint32_t)mask[e + 4 * k + q] << (8 * q);
      w[k] = x;
    }
  }
  uint32_t f = 0;
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    const uint32_t nz = nonzero_bytes(w[k]);  // bits 7, 15, 23, 31
    f |= ((nz >> 7) & 1u) << (4 * k) | ((nz >> 15) & 1u) << (4 * k + 1) |
         ((nz >> 23) & 1u) << (4 * k + 2) | ((nz >> 31) & 1u) << (4 * k + 3);
  }
  return f;
}

// Bit q set when vertex vs + q of a group lies in [0, V) (vs > -16, vs < V).
__device__ __forceinline__ uint32_t in_body_bits(int32_t vs, int32_t V) {
  const int lo = vs < 0 ? -vs : 0;
  const int hi = V - vs < 16 ? V - vs : 16;
  const uint32_t below_hi = hi >= 16 ? 0xFFFFu : ((1u << hi) - 1u);
  return below_hi & ~((1u << lo) - 1u);
}

// Block b takes body b (entries [b*V, (b+1)*V) of the flattened mask).
//   1. its first row is the count of every span of the count kernel before
//      the span holding the body's first entry, plus the active bytes of
//      that span up to the entry; N' is the sum over every span (block 0
//      publishes it, as compact_write_kernel does, before anything else);
//   2. the 16-byte mask groups touching the body, T per pass, one per
//      thread: a block scan of the per-group counts numbers the body's rows;
//      inv and row_ptr[b] are written, and LDS keeps the local row of every
//      vertex (-1 when inactive) and the vertex of every local row;
//   3. a thread per row: its coordinates, and table[j * N' + i] for slots
//      j < K from the neighbour lists and the LDS numbering, written only when
//      N' <= cap (the table holds K rows of cap entries).
// Rows are numbered exactly as compact_write_kernel numbers them, and the
// table entries are those of neighbor_table_kernel.
template <int T, int KM>
__global__ __launch_bounds__(T) void compact_table_kernel(
    const uint8_t* __restrict__ mask, int32_t B, int32_t V, int64_t per_block, int32_t nblocks,
    const int32_t* __restrict__ counts, int32_t* __restrict__ coords, int32_t* __restrict__ inv,
    int32_t* __restrict__ row_ptr, int32_t* __restrict__ n_active, int64_t* n_host, int64_t cap,
    const int32_t* __restrict__ nbr, int32_t K, int32_t* __restrict__ table) {
  constexpr int W = T / 64;
  extern __shared__ int32_t lds_dyn[];
  __shared__ uint32_t red[3 * W];
  __shared__ uint32_t wave_tot[W];
  // local row of vertex v, or -1, at row_l[v + v / 16]: a thread writes the 16
  // vertices of its group, and the padding word spreads the lanes' 16-word
  // strides over every LDS bank
  int32_t* row_l = lds_dyn;                              // [V + V / 16 + 1]
  int32_t* vert_l = lds_dyn + compact_table_row_words(V);  // [V] vertex of local row r
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int b = blockIdx.x;
  const int64_t total_e = (int64_t)B * V;
  const int64_t e0 = (int64_t)b * V, e1 = e0 + V;
  const int64_t g0 = e0 >> 4;
  const int64_t ng = ((e1 + 15) >> 4) - g0;

  // the first pass's mask groups are loaded while the first row is formed
  const __amdgpu_buffer_rsrc_t m_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint8_t*>(mask), (short)0, (int)total_e, kBufferWord3);
  uint32_t wg[4];
  load_group(m_rsrc, g0 + tid, wg);

  // 1. first row of the body, and N'
  const int64_t s0 = e0 / per_block;
  uint32_t before = 0, all = 0, part = 0;
  for (int q = tid; q < nblocks; q += T) {
    const uint32_t c = (uint32_t)counts[q];
    all += c;
    before += q < s0 ? c : 0u;
  }
  for (int64_t p = s0 * per_block + 4 * (int64_t)tid; p < e0; p += 4 * (int64_t)T) {
    uint32_t w = 0;
    if (p + 4 <= total_e) {
      w = *reinterpret_cast<const uint32_t*>(mask + p);
    } else {
      for (int q = 0; q < 4; ++q)
        if (p + q < total_e) w |= (uint32_t)mask[p + q] << (8 * q);
    }
    uint32_t keep = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (p + q < e0) keep |= 0x80u << (8 * q);
    part += (uint32_t)__popc(nonzero_bytes(w) & keep);
  }
  block_sum3<T>(before, all, part, red);
  const int64_t base = (int64_t)before + part;
  const int64_t n_total = all;
  if (tid == 0) {
    if (b == 0) {
      row_ptr[B] = (int32_t)n_total;
      *n_active = (int32_t)n_total;
      // page-locked host copy of the count: a system-scope store
      if (n_host != nullptr)
        __hip_atomic_store(n_host, n_total, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    row_ptr[b] = (int32_t)base;
  }

  // 2. rows of the body (local numbers and vertices fit in 32 bits: V < 2^31)
  int32_t run = 0;  // rows of earlier passes
  const int32_t base32 = (int32_t)base;
  for (int64_t gs = 0; gs < ng; gs += T) {
    const int64_t g = g0 + gs + tid;
    uint32_t cur[4] = {wg[0], wg[1], wg[2], wg[3]};
    load_group(m_rsrc, g + T, wg);  // the next pass's groups (zeros past the mask)
    const bool mine = gs + tid < ng;
    const int32_t vs = (int32_t)(g * 16 - e0);  // vertex of the group's first byte
    uint32_t inb = 0, f = 0;
    if (mine) {
      inb = in_body_bits(vs, V);
      f = group_flags(mask, total_e, cur, g) & inb;
    }
    const uint32_t cnt = (uint32_t)__popc(f);
    const uint32_t inc = wave_inclusive_scan(cnt);
    lds_barrier();  // wave_tot reuse across passes
    if (lane == 63) wave_tot[wave] = inc;
    lds_barrier();
    uint32_t ex = inc - cnt, pass_tot = 0;
#pragma unroll
    for (int q = 0; q < W; ++q) {
      ex += q < wave ? wave_tot[q] : 0u;
      pass_tot += wave_tot[q];
    }
    if (mine) {
      int32_t loc = run + (int32_t)ex;  // local row of the next active entry
      int32_t out[16];
#pragma unroll
      for (int q = 0; q < 16; ++q) {
        const bool on = (f >> q) & 1u;
        const int32_t v = vs + q;
        out[q] = on ? base32 + loc : -1;
        if ((inb >> q) & 1u) row_l[v + (v >> 4)] = on ? loc : -1;
        if (on) vert_l[loc] = v;
        loc += on ? 1 : 0;
      }
      int32_t* dst = inv + g * 16;
      if (inb == 0xFFFFu) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
          *reinterpret_cast<i32x4*>(dst + 4 * k) =
              i32x4{out[4 * k], out[4 * k + 1], out[4 * k + 2], out[4 * k + 3]};
      } else {
#pragma unroll
        for (int q = 0; q < 16; ++q)
          if ((inb >> q) & 1u) dst[q] = out[q];
      }
    }
    run += (int32_t)pass_tot;
  }
  lds_barrier();  // row_l and vert_l complete (the global stores stay in flight)

  // 3. coordinates of the body's rows (one coalesced store per row), and
  // their neighbour-row table
  const bool with_table = table != nullptr && n_total <= cap;
  for (int32_t r = tid; r < run; r += T) {
    const int32_t v = vert_l[r];
    if (base + r < cap) reinterpret_cast<int2*>(coords)[base + r] = make_int2(b, v);
    if (!with_table) continue;
    const int32_t* nrow = nbr + (int64_t)v * K;
    int32_t u[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j) u[j] = nrow[j < K ? j : K - 1];
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (j < K) {
        const int32_t l = (u[j] >= 0 && u[j] < V) ? row_l[u[j] + (u[j] >> 4)] : -1;
        table[(int64_t)j * n_total + base + r] = l >= 0 ? (int32_t)(base + l) : -1;
      }
    }
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


bool compact_table_supported(int32_t V, int32_t K) {
  return V > 0 && V <= kCompactTableMaxV && K > 0 && K <= 32;
}

namespace {
template <int T, int KM>
hipError_t launch_compact_table_k(const uint8_t* mask, int32_t B, int32_t V, int64_t per_block,
                                  int32_t nblocks, const int32_t* counts, int32_t* coords,
                                  int32_t* inv, int32_t* row_ptr, int32_t* n_active,
                                  int64_t* n_host, int64_t cap, const int32_t* nbr, int32_t K,
                                  int32_t* table, hipStream_t stream) {
  auto kern = compact_table_kernel<T, KM>;
  // allow the large dynamic LDS allocation; once per instantiation
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [&] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                   hipFuncAttributeMaxDynamicSharedMemorySize,
                                   compact_table_lds_bytes(kCompactTableMaxV));
  });
  if (attr_err != hipSuccess) return attr_err;
  const size_t lds = (size_t)compact_table_lds_bytes(V);
  hipLaunchKernelGGL(kern, dim3(B), dim3(T), lds, stream, mask, B, V, per_block, nblocks, counts,
                     coords, inv, row_ptr, n_active, n_host, cap, nbr, K, table);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_compact_table(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                                int32_t* inv, int32_t* row_ptr, int32_t* n_active,
                                int64_t* n_host, int64_t cap, const int32_t* nbr, int32_t K,
                                int32_t* table, int32_t* block_counts, hipStream_t stream) {
  const int64_t total = (int64_t)B * V;
  int32_t nblocks;
  int64_t per_block;
  compact_plan(total, &nblocks, &per_block);
  hipLaunchKernelGGL(compact_count_kernel, dim3(nblocks), dim3(kThreads), 0, stream, mask, total,
                     per_block, block_counts);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;
  // one 16-byte group per thread and pass: 1024 threads cover 16 K vertices
  const bool big = V > 4096;
#define SHC_CT_ARGS                                                                          \
  mask, B, V, per_block, nblocks, block_counts, coords, inv, row_ptr, n_active, n_host, cap, \
      nbr, K, table, stream
  if (K <= 10)
    return big ? launch_compact_table_k<1024, 10>(SHC_CT_ARGS)
               : launch_compact_table_k<256, 10>(SHC_CT_ARGS);
  return big ? launch_compact_table_k<1024, 32>(SHC_CT_ARGS)
             : launch_compact_table_k<256, 32>(SHC_CT_ARGS);
#undef SHC_CT_ARGS
}

}  // namespace shc
