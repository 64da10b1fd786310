// Gathered-row contraction on MFMA: the sparse linear layer (Eq. 6) and the
// sparse neighbourhood convolution (Eqs. 4-5), with bias and activation
// (Eq. 10) fused into the epilogue.
//
// Both are one product over a flattened reduction axis kk = j * Cin + c:
//
//   out[i][n] = act( bias[n] + sum_kk A[i][kk] * W[kk][n] ),
//   A[i][j*Cin + c] = S[r_ij][c]  (zero when r_ij = -1),
//
// where W is the caller's [K][Cin][Cout] array read as [K*Cin][Cout], and
// r_ij = i for the linear layer (K = 1) or inv[b_i*V + nbr[v_i*K + j]] for the
// convolution.  Concatenating the slots this way is the spiral-convolution
// form of Eqs. 4-5: row i of A is the neighbourhood of active vertex i, and
// the per-output index list r_i. is the paper's indexing matrix (Eq. 4)
// evaluated on the fly.
//
// Tiling (one workgroup = 4 wavefronts = 256 threads):
//   * a tile of BM = 128 active rows x BN (64 or 128) output channels; tiles
//     are handed out so that each XCD works on a contiguous range of rows
//     (neighbour rows of one body then stay in that XCD's L2);
//   * the tile's index lists are built with all loads of one level in flight
//     at once (coordinates, then neighbour vertices, then inverse-map rows);
//   * wavefronts in a 2 x 2 grid, each owning 64 rows x BN/2 columns as
//     16 x 16 MFMA blocks (v_mfma_f32_16x16x32_bf16 for bf16 inputs,
//     v_mfma_f32_16x16x4_f32 for fp32) with fp32 accumulators;
//   * the reduction axis advances in chunks of 64 bytes per row (32 bf16 or
//     16 fp32 entries, one MFMA k-step).  Global loads run two chunks ahead
//     in registers; a chunk of A (gathered neighbour rows, row-major) and of
//     W (natural [k][n] layout) is copied to one of two LDS buffers while the
//     MFMAs read the other, with one barrier per chunk;
//   * bf16 B fragments are read from the [k][n] LDS layout with the gfx950
//     transposing load ds_read_b64_tr_b16 (two per fragment), so W is never
//     transposed in registers; fp32 B fragments are single dwords;
//   * absent neighbour rows are written to LDS as zeros without a global
//     load; a 16-row MFMA block whose rows have no present neighbour in the
//     slot(s) of a chunk is skipped (its product would be zero), and so is a
//     chunk that no row of the tile needs;
//   * the epilogue adds the bias, applies the activation, rounds to the
//     output dtype and writes whole rows through LDS as 16-byte vectors.
//
// MFMA operand layout (CDNA3/CDNA4, 64 lanes, g = lane / 16, i = lane % 16):
//   A block 16 x k: lane (g, i) supplies row i, k-group g;
//   B block k x 16: lane (g, i) supplies column i, k-group g;
//   D block 16 x 16: lane (g, i) holds rows 4g .. 4g+3 of column i.
// A and B use the same k-group -> k mapping, so the order in which the
// hardware walks k inside a group does not change the result.
#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kThreads = 256;
constexpr int BM = 128;
constexpr int kRowBlocks = BM / 16;
constexpr int kChunkBytes = 64;            // reduction bytes per row per chunk (one k-step)
constexpr int kARow = kChunkBytes + 16;    // padded LDS row of the A stage (bytes)
constexpr int kMaxSlots = 32;
constexpr int kSlotsPerThread = kMaxSlots / 2;  // two threads build one row's index list

typedef __bf16 bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
#define SHC_LDS __attribute__((address_space(3)))

template <bool BF16>
struct Elem;
template <>
struct Elem<true> {
  static constexpr int bytes = 2;
  static constexpr int per_vec = 8;  // elements per 16 bytes
};
template <>
struct Elem<false> {
  static constexpr int bytes = 4;
  static constexpr int per_vec = 4;
};

template <bool BF16, int BN>
struct Layout {
  using E = Elem<BF16>;
  static constexpr int KC = kChunkBytes / E::bytes;   // reduction entries per chunk
  static constexpr int WRow = BN * E::bytes + 16;      // padded LDS row of the W stage
  static constexpr int AStage = BM * kARow;
  static constexpr int WStage = KC * WRow;
  static constexpr int Stage = AStage + WStage;
  static constexpr int ORow = BN * E::bytes + 16;      // padded LDS row of the output stage
  static constexpr int OutHalf = (BM / 2) * ORow;      // epilogue writes 64 rows at a time
  static constexpr int Main = (2 * Stage > OutHalf) ? 2 * Stage : OutHalf;
  static constexpr int AVecPerRow = kChunkBytes / 16;
  static constexpr int AVecs = BM * AVecPerRow / kThreads;  // per thread
  static constexpr int WVecPerRow = BN * E::bytes / 16;
  static constexpr int WVecs = (KC * WVecPerRow + kThreads - 1) / kThreads;
};

template <int BN, bool BF16>
size_t lds_bytes(int K) {
  return (size_t)Layout<BF16, BN>::Main + (size_t)BM * K * sizeof(int32_t) +
         kRowBlocks * sizeof(uint32_t) + 2 * BM * sizeof(int32_t);
}

// (slot, offset) of reduction entry `off` entries past (j, c)
__device__ __forceinline__ void advance(int& j, int& c, int off, int Cin) {
  c += off;
  while (c >= Cin) {
    c -= Cin;
    ++j;
  }
}

__device__ __forceinline__ uint32_t slot_range_bits(int j0, int j1) {
  const uint32_t upto = (j1 >= 31) ? 0xFFFFFFFFu : ((2u << j1) - 1u);
  return upto & ~((1u << j0) - 1u);
}

template <bool BF16, int BN, bool CONV>
__global__ __launch_bounds__(kThreads, 3) void gather_gemm_kernel(GemmArgs a) {
  using E = Elem<BF16>;
  using Lt = Layout<BF16, BN>;
  constexpr int KC = Lt::KC;
  constexpr int WN = BN / 2;   // columns per wavefront
  constexpr int NB = WN / 16;  // 16-column blocks per wavefront

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int K = CONV ? a.K : 1;
  int32_t* srcs = reinterpret_cast<int32_t*>(smem + Lt::Main);        // [BM][K]
  uint32_t* blk_slots = reinterpret_cast<uint32_t*>(srcs + BM * K);    // [BM/16]
  int32_t* row_b = reinterpret_cast<int32_t*>(blk_slots + kRowBlocks);  // [BM]
  int32_t* row_v = row_b + BM;                                         // [BM]

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int g = lane >> 4;
  const int l16 = lane & 15;

  // XCD-aware tile order: workgroup b runs on XCD b % 8; give each XCD a
  // contiguous range of row tiles.
  const int ntiles = gridDim.x;
  const int bid = blockIdx.x;
  const int per_xcd = ntiles / 8;
  const int rem = ntiles % 8;
  const int xcd = bid % 8;
  const int slot_in_xcd = bid / 8;
  const int tile =
      (xcd < rem ? xcd * (per_xcd + 1) : rem * (per_xcd + 1) + (xcd - rem) * per_xcd) +
      slot_in_xcd;

  const int64_t row0 = (int64_t)tile * BM;
  const int n0 = blockIdx.y * BN;
  const int Cin = a.Cin;
  const int Cout = a.Cout;
  const int Ktot = K * Cin;
  const int nchunks = (Ktot + KC - 1) / KC;
  const unsigned char* S = static_cast<const unsigned char*>(a.S);
  const unsigned char* W = static_cast<const unsigned char*>(a.W);

  // ---- index lists of the tile -----------------------------------------------
  if (tid < kRowBlocks) blk_slots[tid] = 0;
  if (CONV) {
    if (tid < BM) {
      const int64_t i = row0 + tid;
      int b = -1, v = -1;
      if (i < a.n_rows) {
        const int2 c = reinterpret_cast<const int2*>(a.coords)[i];
        if (c.x >= 0 && c.x < a.B && c.y >= 0 && c.y < a.V) {
          b = c.x;
          v = c.y;
        }
      }
      row_b[tid] = b;
      row_v[tid] = v;
    }
    __syncthreads();
    // two threads per row; thread h of row r takes slots h, h + 2, h + 4, ...
    const int r = tid >> 1;
    const int h = tid & 1;
    const int b = row_b[r];
    const int v = row_v[r];
    int32_t nb[kSlotsPerThread];
#pragma unroll
    for (int m = 0; m < kSlotsPerThread; ++m) {
      const int j = h + 2 * m;
      nb[m] = -1;
      if (j < K && v >= 0) nb[m] = a.nbr[(int64_t)v * K + j];
    }
    uint32_t bits = 0;
#pragma unroll
    for (int m = 0; m < kSlotsPerThread; ++m) {
      const int j = h + 2 * m;
      int32_t src = -1;
      if (j < K && nb[m] >= 0 && nb[m] < a.V) {
        const int32_t s = a.inv[(int64_t)b * a.V + nb[m]];
        if (s >= 0 && (int64_t)s < a.n_rows) src = s;
      }
      if (j < K) srcs[r * K + j] = src;
      if (src >= 0) bits |= 1u << j;
    }
    __syncthreads();  // blk_slots cleared above before any atomic
    if (bits) atomicOr(&blk_slots[r >> 4], bits);
  } else {
    __syncthreads();
    if (tid < BM) {
      const int64_t i = row0 + tid;
      srcs[tid] = i < a.n_rows ? (int32_t)i : -1;
      if (i < a.n_rows) atomicOr(&blk_slots[tid >> 4], 1u);
    }
  }
  __syncthreads();
  uint32_t tile_slots = 0;
#pragma unroll
  for (int q = 0; q < kRowBlocks; ++q) tile_slots |= blk_slots[q];
  uint32_t my_blk[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb) my_blk[rb] = blk_slots[wm * 4 + rb];

  // ---- chunk bookkeeping (no division in the loop) ---------------------------
  // A chunk starts at reduction entry k0 = chunk * KC, i.e. slot js, offset cs.
  struct Pos {
    int chunk, js, cs;
  };
  auto chunk_bits = [&](const Pos& p) -> uint32_t {
    int je = p.js, ce = p.cs;
    advance(je, ce, min(KC, Ktot - p.chunk * KC) - 1, Cin);
    return slot_range_bits(p.js, je);
  };
  // first live chunk at or after p (p.chunk == nchunks when none)
  auto next_live = [&](Pos p) -> Pos {
    while (p.chunk < nchunks && (chunk_bits(p) & tile_slots) == 0u) {
      ++p.chunk;
      advance(p.js, p.cs, KC, Cin);
    }
    return p;
  };
  auto step = [&](Pos p) -> Pos {
    ++p.chunk;
    advance(p.js, p.cs, KC, Cin);
    return next_live(p);
  };

  // ---- global -> register -> LDS staging -------------------------------------
  struct Regs {
    i32x4 a[Lt::AVecs];
    i32x4 w[Lt::WVecs];
  };

  auto load_chunk = [&](const Pos& p, Regs& R) {
    const int k0 = p.chunk * KC;
#pragma unroll
    for (int u = 0; u < Lt::AVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int r = idx / Lt::AVecPerRow;
      const int q = idx % Lt::AVecPerRow;
      int j = p.js, c = p.cs;
      advance(j, c, q * E::per_vec, Cin);
      i32x4 v = {0, 0, 0, 0};
      if (k0 + q * E::per_vec < Ktot) {
        const int32_t src = srcs[r * K + j];
        if (src >= 0)
          v = *reinterpret_cast<const i32x4*>(S + ((int64_t)src * Cin + c) * E::bytes);
      }
      R.a[u] = v;
    }
#pragma unroll
    for (int u = 0; u < Lt::WVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int kr = idx / Lt::WVecPerRow;
      const int q = idx % Lt::WVecPerRow;
      const int kk = k0 + kr;
      const int n = n0 + q * E::per_vec;
      i32x4 v = {0, 0, 0, 0};
      if (kr < KC && kk < Ktot && n < Cout)
        v = *reinterpret_cast<const i32x4*>(W + ((int64_t)kk * Cout + n) * E::bytes);
      R.w[u] = v;
    }
  };

  auto store_chunk = [&](const Regs& R, int buf) {
    unsigned char* a_lds = smem + buf * Lt::Stage;
    unsigned char* w_lds = a_lds + Lt::AStage;
#pragma unroll
    for (int u = 0; u < Lt::AVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int r = idx / Lt::AVecPerRow;
      const int q = idx % Lt::AVecPerRow;
      *reinterpret_cast<i32x4*>(a_lds + r * kARow + q * 16) = R.a[u];
    }
#pragma unroll
    for (int u = 0; u < Lt::WVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int kr = idx / Lt::WVecPerRow;
      const int q = idx % Lt::WVecPerRow;
      if (kr < KC) *reinterpret_cast<i32x4*>(w_lds + kr * Lt::WRow + q * 16) = R.w[u];
    }
  };

  f32x4 acc[4][NB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const Pos& p, int buf) {
    const unsigned char* a_lds = smem + buf * Lt::Stage;
    const unsigned char* w_lds = a_lds + Lt::AStage;
    const uint32_t bits = chunk_bits(p);
    if (BF16) {
      bf16x8 bfrag[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        // k rows 8g + (0..3 | 4..7), columns cb*16 + 4*(l16 % 4) of this lane's group
        const int col = wn * WN + cb * 16 + 4 * (l16 & 3);
        const int kr = 8 * g + (l16 >> 2);
        const unsigned char* p0 = w_lds + kr * Lt::WRow + col * 2;
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0)));
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
            (SHC_LDS bf16x4*)(const_cast<unsigned char*>(p0 + 4 * Lt::WRow)));
        bfrag[cb] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
      }
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if ((my_blk[rb] & bits) == 0u) continue;
        const int row = wm * 64 + rb * 16 + l16;
        const i32x4 af = *reinterpret_cast<const i32x4*>(a_lds + row * kARow + g * 16);
        const bf16x8 afrag = __builtin_bit_cast(bf16x8, af);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
          acc[rb][cb] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag, bfrag[cb], acc[rb][cb], 0, 0, 0);
      }
    } else {
      // fp32: lane group g holds k = 4g .. 4g+3 of this 16-entry chunk;
      // MFMA s uses component s of the A vector and W row 4g + s.
      float bw[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const int col = wn * WN + cb * 16 + l16;
#pragma unroll
        for (int s = 0; s < 4; ++s)
          bw[cb][s] = *reinterpret_cast<const float*>(w_lds + (4 * g + s) * Lt::WRow + col * 4);
      }
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if ((my_blk[rb] & bits) == 0u) continue;
        const int row = wm * 64 + rb * 16 + l16;
        const i32x4 af = *reinterpret_cast<const i32x4*>(a_lds + row * kARow + g * 16);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int s = 0; s < 4; ++s)
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(__int_as_float(af[s]), bw[cb][s],
                                                               acc[rb][cb], 0, 0, 0);
      }
    }
  };

  // ---- main loop: loads two chunks ahead, LDS double buffer -------------------
  // Invariant at the top of an iteration: chunk `c0` is in LDS buffer `buf`,
  // chunk `c1` (the next live one) is in registers R[x] (or absent), and R[x^1]
  // is free.
  Regs R0, R1;
  Pos c0 = next_live(Pos{0, 0, 0});
  Pos c1 = c0.chunk < nchunks ? step(c0) : c0;
  if (c0.chunk < nchunks) {
    load_chunk(c0, R0);
    if (c1.chunk < nchunks) load_chunk(c1, R1);
    store_chunk(R0, 0);
  }
  __syncthreads();
  int buf = 0;
  // two iterations per trip so that the register sets keep fixed roles
  while (c0.chunk < nchunks) {
    {
      const Pos c2 = c1.chunk < nchunks ? step(c1) : c1;
      if (c2.chunk < nchunks) load_chunk(c2, R0);
      compute(c0, buf);
      if (c1.chunk < nchunks) store_chunk(R1, buf ^ 1);
      __syncthreads();
      buf ^= 1;
      c0 = c1;
      c1 = c2;
    }
    if (c0.chunk >= nchunks) break;
    {
      const Pos c2 = c1.chunk < nchunks ? step(c1) : c1;
      if (c2.chunk < nchunks) load_chunk(c2, R1);
      compute(c0, buf);
      if (c1.chunk < nchunks) store_chunk(R0, buf ^ 1);
      __syncthreads();
      buf ^= 1;
      c0 = c1;
      c1 = c2;
    }
  }

  // ---- epilogue: bias + activation + rounding, staged through LDS -----------
  // rows 0..63 (wm = 0) first, then rows 64..127 (wm = 1)
  unsigned char* o_lds = smem;
  unsigned char* out = static_cast<unsigned char*>(a.out);
  constexpr int kVecPerRow = BN * E::bytes / 16;
  const int ncols = min(BN, Cout - n0);
  const int vec_valid = ncols * E::bytes / 16;
  for (int half = 0; half < 2; ++half) {
    if (wm == half) {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const int col_l = wn * WN + cb * 16 + l16;
        const int col = n0 + col_l;
        const float bv = (a.bias != nullptr && col < Cout) ? a.bias[col] : 0.f;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row_l = rb * 16 + g * 4 + r;
            float v = acc[rb][cb][r] + bv;
            if (a.relu) v = v > 0.f ? v : 0.f;
            unsigned char* p = o_lds + row_l * Lt::ORow + col_l * E::bytes;
            if (BF16)
              *reinterpret_cast<uint16_t*>(p) = (uint16_t)f32_to_bf16_bits(v);
            else
              *reinterpret_cast<float*>(p) = v;
          }
        }
      }
    }
    __syncthreads();
    for (int idx = tid; idx < (BM / 2) * kVecPerRow; idx += kThreads) {
      const int r = idx / kVecPerRow;
      const int q = idx % kVecPerRow;
      const int64_t i = row0 + half * (BM / 2) + r;
      if (i < a.n_rows && q < vec_valid) {
        const i32x4 v = *reinterpret_cast<const i32x4*>(o_lds + r * Lt::ORow + q * 16);
        *reinterpret_cast<i32x4*>(out + (i * Cout + n0) * E::bytes + q * 16) = v;
      }
    }
    __syncthreads();
  }
}

template <bool BF16, int BN, bool CONV>
hipError_t launch_tile(const GemmArgs& a, hipStream_t stream) {
  const unsigned gx = (unsigned)((a.n_rows + BM - 1) / BM);
  const unsigned gy = (unsigned)((a.Cout + BN - 1) / BN);
  const size_t lds = lds_bytes<BN, BF16>(CONV ? a.K : 1);
  auto kern = gather_gemm_kernel<BF16, BN, CONV>;
  // allow more than 64 KB of dynamic LDS (gfx950 has 160 KB per CU); once per instantiation
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [&] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, 160 * 1024);
  });
  if (attr_err != hipSuccess) return attr_err;
  hipLaunchKernelGGL(kern, dim3(gx, gy), dim3(kThreads), lds, stream, a);
  return hipGetLastError();
}

template <bool BF16, bool CONV>
hipError_t launch_typed(const GemmArgs& a, hipStream_t stream) {
  if (a.Cout >= 128) return launch_tile<BF16, 128, CONV>(a, stream);
  return launch_tile<BF16, 64, CONV>(a, stream);
}

}  // namespace

hipError_t launch_gather_gemm(const GemmArgs& a, bool conv, bool bf16, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  if (bf16) return conv ? launch_typed<true, true>(a, stream) : launch_typed<true, false>(a, stream);
  return conv ? launch_typed<false, true>(a, stream) : launch_typed<false, false>(a, stream);
}

}  // namespace shc
