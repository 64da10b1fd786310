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
// form of Eqs. 4-5: row i of A is the neighbourhood of active vertex i.
//
// Tiling (one workgroup = 4 wavefronts = 256 threads):
//   * a tile of BM = 64 active rows x BN (64 or 128) output channels;
//   * wavefronts in a 2 x 2 grid, each owning 32 rows x BN/2 columns as
//     16 x 16 MFMA blocks (v_mfma_f32_16x16x32_bf16 for bf16 inputs,
//     v_mfma_f32_16x16x4_f32 for fp32, fp32 accumulators);
//   * the reduction axis advances in chunks of 128 bytes per row (64 bf16 or
//     32 fp32 entries).  A chunk of A (the gathered neighbour rows) and the
//     matching chunk of W, transposed so that every lane reads 16 contiguous
//     bytes of one column, are staged in LDS; the next chunk's global loads
//     are issued before the MFMAs of the current one;
//   * neighbour rows that are absent are written to LDS as zeros without a
//     global load, and a 16-row MFMA block whose rows have no present
//     neighbour for the slot(s) of a k-step is skipped (its product is zero);
//   * the epilogue adds the bias, applies the activation, rounds to the
//     output dtype and writes whole rows through LDS as 16-byte vectors.
//
// MFMA operand layout used below (CDNA3/CDNA4, 64 lanes, g = lane / 16):
//   A block 16 x k: lane (g, i = lane % 16) supplies row i, k-group g;
//   B block k x 16: lane (g, j = lane % 16) supplies column j, k-group g;
//   D block 16 x 16: lane (g, j) holds rows 4g .. 4g+3 of column j.
// The same k-group -> k mapping is used for A and B, so the order in which
// the hardware walks k inside a group does not change the result.
#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kThreads = 256;
constexpr int BM = 64;
constexpr int kChunkBytes = 128;              // reduction bytes per row per chunk
constexpr int kRowStride = kChunkBytes + 16;  // padded LDS row (bytes), conflict-free b128 reads
constexpr int kMaxK = 32;

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

// 8 x 8 transpose of 16-bit values: in[k] holds row k (columns 0..7, two per
// dword); out[n] receives column n (rows 0..7).
__device__ __forceinline__ void transpose8x8_b16(const i32x4 in[8], i32x4 out[8]) {
#pragma unroll
  for (int n = 0; n < 8; ++n) {
    const int wsel = n >> 1;
    const int sh = (n & 1) * 16;
    uint32_t w[4];
#pragma unroll
    for (int p = 0; p < 4; ++p) {
      const uint32_t a = ((uint32_t)in[2 * p][wsel] >> sh) & 0xFFFFu;
      const uint32_t b = ((uint32_t)in[2 * p + 1][wsel] >> sh) & 0xFFFFu;
      w[p] = a | (b << 16);
    }
    out[n] = i32x4{(int)w[0], (int)w[1], (int)w[2], (int)w[3]};
  }
}

__device__ __forceinline__ void transpose4x4_b32(const i32x4 in[4], i32x4 out[4]) {
#pragma unroll
  for (int n = 0; n < 4; ++n) out[n] = i32x4{in[0][n], in[1][n], in[2][n], in[3][n]};
}

template <bool BF16, int BN, bool CONV>
__global__ __launch_bounds__(kThreads) void gather_gemm_kernel(GemmArgs a) {
  using E = Elem<BF16>;
  constexpr int KC = kChunkBytes / E::bytes;  // reduction entries per chunk
  constexpr int WN = BN / 2;                  // columns per wavefront
  constexpr int NB = WN / 16;                 // 16-column blocks per wavefront
  constexpr int kOutStride = BN * E::bytes + 16;
  constexpr int kStageBytes = (BM + BN) * kRowStride;
  constexpr int kOutBytes = BM * kOutStride;
  constexpr int kLdsBytes = kStageBytes > kOutBytes ? kStageBytes : kOutBytes;

  __shared__ __attribute__((aligned(16))) unsigned char lds[kLdsBytes];
  __shared__ int32_t srcs[BM * kMaxK];
  __shared__ uint32_t blk_slots[BM / 16];  // bit j: some row of the 16-row block has slot j present

  unsigned char* a_lds = lds;
  unsigned char* w_lds = lds + BM * kRowStride;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave & 1;
  const int wn = wave >> 1;
  const int g = lane >> 4;
  const int l16 = lane & 15;

  const int64_t row0 = (int64_t)blockIdx.x * BM;
  const int n0 = blockIdx.y * BN;
  const int K = CONV ? a.K : 1;
  const int Cin = a.Cin;
  const int Cout = a.Cout;
  const int Ktot = K * Cin;
  const int nchunks = (Ktot + KC - 1) / KC;
  const unsigned char* S = static_cast<const unsigned char*>(a.S);
  const unsigned char* W = static_cast<const unsigned char*>(a.W);

  // ---- source rows of the tile ------------------------------------------
  if (tid < BM / 16) blk_slots[tid] = 0;
  __syncthreads();
  for (int e = tid; e < BM * K; e += kThreads) {
    const int r = e / K;
    const int j = e - r * K;
    const int64_t i = row0 + r;
    int32_t src = -1;
    if (i < a.n_rows) {
      if (CONV) {
        const int2 c = reinterpret_cast<const int2*>(a.coords)[i];
        if (c.x >= 0 && c.x < a.B && c.y >= 0 && c.y < a.V) {
          const int32_t nb = a.nbr[(int64_t)c.y * K + j];
          if (nb >= 0 && nb < a.V) {
            const int32_t s = a.inv[(int64_t)c.x * a.V + nb];
            if (s >= 0 && (int64_t)s < a.n_rows) src = s;
          }
        }
      } else {
        src = (int32_t)i;
      }
    }
    srcs[r * K + j] = src;
    if (src >= 0) atomicOr(&blk_slots[r >> 4], 1u << j);
  }
  __syncthreads();
  uint32_t tile_slots = 0;
#pragma unroll
  for (int q = 0; q < BM / 16; ++q) tile_slots |= blk_slots[q];

  // slots touched by reduction entries [k_lo, k_hi)
  auto slot_bits = [&](int k_lo, int k_hi) -> uint32_t {
    if (k_lo >= Ktot) return 0u;
    const int j0 = k_lo / Cin;
    const int j1 = (min(k_hi, Ktot) - 1) / Cin;
    const uint32_t upto = (j1 >= 31) ? 0xFFFFFFFFu : ((2u << j1) - 1u);
    return upto & ~((1u << j0) - 1u);
  };

  // ---- global -> register staging ----------------------------------------
  // A: BM rows x 8 vectors of 16 bytes; 2 vectors per thread.
  constexpr int kAVecs = BM * (kChunkBytes / 16) / kThreads;
  // W: transposed sub-blocks; bf16 8(k) x 8(n), fp32 4(k) x 4(n).
  constexpr int SUBK = BF16 ? 8 : 4;
  constexpr int SUBN = BF16 ? 8 : 4;
  constexpr int kWSub = (KC / SUBK) * (BN / SUBN);
  constexpr int kWIters = (kWSub + kThreads - 1) / kThreads;

  i32x4 a_reg[kAVecs];
  i32x4 w_reg[kWIters][SUBK];

  auto load_chunk = [&](int chunk) {
    const int k0 = chunk * KC;
#pragma unroll
    for (int u = 0; u < kAVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int r = idx >> 3;
      const int q = idx & 7;
      const int kk = k0 + q * E::per_vec;
      i32x4 v = {0, 0, 0, 0};
      if (kk < Ktot) {
        const int j = kk / Cin;
        const int c = kk - j * Cin;
        const int32_t src = srcs[r * K + j];
        if (src >= 0)
          v = *reinterpret_cast<const i32x4*>(S + ((int64_t)src * Cin + c) * E::bytes);
      }
      a_reg[u] = v;
    }
#pragma unroll
    for (int it = 0; it < kWIters; ++it) {
      const int sb = tid + it * kThreads;
      const int sk = sb % (KC / SUBK);
      const int sn = sb / (KC / SUBK);
      const int n = n0 + sn * SUBN;
#pragma unroll
      for (int t = 0; t < SUBK; ++t) {
        const int kk = k0 + sk * SUBK + t;
        i32x4 v = {0, 0, 0, 0};
        if (sb < kWSub && kk < Ktot && n < Cout)
          v = *reinterpret_cast<const i32x4*>(W + ((int64_t)kk * Cout + n) * E::bytes);
        w_reg[it][t] = v;
      }
    }
  };

  auto store_chunk = [&]() {
#pragma unroll
    for (int u = 0; u < kAVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int r = idx >> 3;
      const int q = idx & 7;
      *reinterpret_cast<i32x4*>(a_lds + r * kRowStride + q * 16) = a_reg[u];
    }
#pragma unroll
    for (int it = 0; it < kWIters; ++it) {
      const int sb = tid + it * kThreads;
      if (sb < kWSub) {
        const int sk = sb % (KC / SUBK);
        const int sn = sb / (KC / SUBK);
        i32x4 tr[SUBN];
        if (BF16)
          transpose8x8_b16(w_reg[it], tr);
        else
          transpose4x4_b32(w_reg[it], tr);
#pragma unroll
        for (int t = 0; t < SUBN; ++t)
          *reinterpret_cast<i32x4*>(w_lds + (sn * SUBN + t) * kRowStride + sk * 16) = tr[t];
      }
    }
  };

  // ---- main loop -------------------------------------------------------
  f32x4 acc[2][NB];
#pragma unroll
  for (int rb = 0; rb < 2; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb) acc[rb][cb] = f32x4{0.f, 0.f, 0.f, 0.f};

  // chunks whose slots are absent from the whole tile contribute nothing
  auto chunk_live = [&](int chunk) -> bool {
    return (slot_bits(chunk * KC, chunk * KC + KC) & tile_slots) != 0u;
  };

  int cur = 0;
  while (cur < nchunks && !chunk_live(cur)) ++cur;
  if (cur < nchunks) {
    load_chunk(cur);
    store_chunk();
  }
  __syncthreads();
  while (cur < nchunks) {
    int nxt = cur + 1;
    while (nxt < nchunks && !chunk_live(nxt)) ++nxt;
    if (nxt < nchunks) load_chunk(nxt);

    const int k0 = cur * KC;
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {  // two 64-byte k-steps per 128-byte chunk
      // entries of this k-step: bf16 32, fp32 16
      const int klo = k0 + ks * (KC / 2);
      const uint32_t bits = slot_bits(klo, klo + KC / 2);
      i32x4 bfrag[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const int col = wn * WN + cb * 16 + l16;
        bfrag[cb] = *reinterpret_cast<const i32x4*>(w_lds + col * kRowStride + ks * 64 + g * 16);
      }
#pragma unroll
      for (int rb = 0; rb < 2; ++rb) {
        if ((blk_slots[wm * 2 + rb] & bits) == 0u) continue;
        const int row = wm * 32 + rb * 16 + l16;
        const i32x4 afrag =
            *reinterpret_cast<const i32x4*>(a_lds + row * kRowStride + ks * 64 + g * 16);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb) {
          if (BF16) {
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, afrag), __builtin_bit_cast(bf16x8, bfrag[cb]),
                acc[rb][cb], 0, 0, 0);
          } else {
#pragma unroll
            for (int s = 0; s < 4; ++s)
              acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                  __int_as_float(afrag[s]), __int_as_float(bfrag[cb][s]), acc[rb][cb], 0, 0, 0);
          }
        }
      }
    }
    __syncthreads();
    if (nxt < nchunks) {
      store_chunk();
      __syncthreads();
    }
    cur = nxt;
  }

  // ---- epilogue: bias + activation + rounding, staged through LDS -------
  unsigned char* o_lds = lds;
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) {
    const int col_l = wn * WN + cb * 16 + l16;
    const int col = n0 + col_l;
    const float bv = (a.bias != nullptr && col < Cout) ? a.bias[col] : 0.f;
#pragma unroll
    for (int rb = 0; rb < 2; ++rb) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int row_l = wm * 32 + rb * 16 + g * 4 + r;
        float v = acc[rb][cb][r] + bv;
        if (a.relu) v = v > 0.f ? v : 0.f;
        unsigned char* p = o_lds + row_l * kOutStride + col_l * E::bytes;
        if (BF16)
          *reinterpret_cast<uint16_t*>(p) = (uint16_t)f32_to_bf16_bits(v);
        else
          *reinterpret_cast<float*>(p) = v;
      }
    }
  }
  __syncthreads();
  constexpr int kVecPerRow = BN * E::bytes / 16;
  const int ncols = min(BN, Cout - n0);
  const int vec_valid = ncols * E::bytes / 16;
  unsigned char* out = static_cast<unsigned char*>(a.out);
  for (int idx = tid; idx < BM * kVecPerRow; idx += kThreads) {
    const int r = idx / kVecPerRow;
    const int q = idx - r * kVecPerRow;
    const int64_t i = row0 + r;
    if (i < a.n_rows && q < vec_valid) {
      const i32x4 v = *reinterpret_cast<const i32x4*>(o_lds + r * kOutStride + q * 16);
      *reinterpret_cast<i32x4*>(out + (i * Cout + n0) * E::bytes + q * 16) = v;
    }
  }
}

template <bool BF16, bool CONV>
hipError_t launch_typed(const GemmArgs& a, hipStream_t stream) {
  const unsigned gx = (unsigned)((a.n_rows + BM - 1) / BM);
  if (a.Cout >= 128) {
    const unsigned gy = (unsigned)((a.Cout + 127) / 128);
    hipLaunchKernelGGL((gather_gemm_kernel<BF16, 128, CONV>), dim3(gx, gy), dim3(kThreads), 0,
                       stream, a);
  } else {
    const unsigned gy = (unsigned)((a.Cout + 63) / 64);
    hipLaunchKernelGGL((gather_gemm_kernel<BF16, 64, CONV>), dim3(gx, gy), dim3(kThreads), 0,
                       stream, a);
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_gather_gemm(const GemmArgs& a, bool conv, bool bf16, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  if (bf16) return conv ? launch_typed<true, true>(a, stream) : launch_typed<true, false>(a, stream);
  return conv ? launch_typed<false, true>(a, stream) : launch_typed<false, false>(a, stream);
}

}  // namespace shc
