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
//   * the accumulators start at the bias; the epilogue applies the activation, rounds to the
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
constexpr int kMaxSlots = 32;

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

template <bool BF16, int BN, int CHUNK, int STAGES>
struct Layout {
  using E = Elem<BF16>;
  static constexpr int KC = CHUNK / E::bytes;          // reduction entries per chunk
  static constexpr int KSTEP = 64 / E::bytes;          // entries per MFMA k-step (64 bytes)
  static constexpr int ARow = CHUNK + 16;              // padded LDS row of the A stage
  static constexpr int WRow = BN * E::bytes + 16;      // padded LDS row of the W stage
  static constexpr int AStage = BM * ARow;
  static constexpr int WStage = KC * WRow;
  static constexpr int Stage = AStage + WStage;
  static constexpr int ORow = BN * E::bytes + 16;      // padded LDS row of the output stage
  static constexpr int Out = BM * ORow;                // whole output tile
  static constexpr int OutHalf = (BM / 2) * ORow;      // half of it
  static constexpr int Main = (STAGES * Stage > OutHalf) ? STAGES * Stage : OutHalf;
  static constexpr bool OnePassOut = Out <= Main;      // else the epilogue runs in two halves
  static constexpr int AVecPerRow = CHUNK / 16;
  static constexpr int AVecs = BM * AVecPerRow / kThreads;  // per thread
  static constexpr int WVecPerRow = BN * E::bytes / 16;
  static constexpr int WVecs = (KC * WVecPerRow + kThreads - 1) / kThreads;
};

// Index area after the staging buffers (int32 words):
//   srcs[BM*K] (row-major in tile order), srcs_p[BM*K] (permuted order),
//   row_b[BM], row_v[BM], rowmask[BM], perm[BM], blk_slots[BM/16],
//   bcnt[2][kMaxSlots + 2], scnt[2][kMaxSlots]
constexpr int kBuckets = kMaxSlots + 2;
inline size_t index_words(int K) {
  return 2 * (size_t)BM * K + 4 * BM + kRowBlocks + 2 * kBuckets + 2 * kMaxSlots;
}

template <bool BF16, int BN, int CHUNK, int STAGES>
size_t lds_bytes(int K) {
  return (size_t)Layout<BF16, BN, CHUNK, STAGES>::Main + index_words(K) * sizeof(int32_t);
}

__device__ __forceinline__ uint32_t slot_range_bits(int j0, int j1) {
  const uint32_t upto = (j1 >= 31) ? 0xFFFFFFFFu : ((2u << j1) - 1u);
  return upto & ~((1u << j0) - 1u);
}

// SPT: neighbour slots per thread when building the index lists (two threads
// per row), a bound on (K + 1) / 2 fixed at compile time.
template <bool BF16, int BN, bool CONV, bool TBL, int CHUNK, int STAGES, int SPT>
__global__ __launch_bounds__(kThreads, 2) void gather_gemm_kernel(GemmArgs a) {
  using E = Elem<BF16>;
  using Lt = Layout<BF16, BN, CHUNK, STAGES>;
  constexpr int KC = Lt::KC;
  constexpr int WN = BN / 2;   // columns per wavefront
  constexpr int NB = WN / 16;  // 16-column blocks per wavefront

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int K = CONV ? a.K : 1;
  int32_t* srcs0 = reinterpret_cast<int32_t*>(smem + Lt::Main);  // [BM][K], tile order
  int32_t* srcs = srcs0 + BM * K;                                // [BM][K], permuted order
  int32_t* row_b = srcs + BM * K;                                // [BM]
  int32_t* row_v = row_b + BM;                                   // [BM]
  uint32_t* rowmask = reinterpret_cast<uint32_t*>(row_v + BM);   // [BM]
  int32_t* perm = reinterpret_cast<int32_t*>(rowmask + BM);      // [BM] tile row at position p
  uint32_t* blk_slots = reinterpret_cast<uint32_t*>(perm + BM);  // [BM/16]
  int32_t* bcnt = reinterpret_cast<int32_t*>(blk_slots + kRowBlocks);  // [2][kBuckets]
  int32_t* scnt = bcnt + 2 * kBuckets;                                 // [2][kMaxSlots]

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
  if (tid < BM) rowmask[tid] = 0;
  if (CONV) {
    // two threads per row; thread h of row r takes slots h, h + 2, h + 4, ...
    const int r = tid >> 1;
    const int h = tid & 1;
    uint32_t bits = 0;
    if (TBL) {
      // one round of loads from the slot-major neighbour-row table
      const bool in = row0 + r < a.n_rows;
      const int64_t i = in ? row0 + r : 0;
      int32_t sv[SPT];
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int j = h + 2 * m;
        sv[m] = a.table[(int64_t)(j < K ? j : K - 1) * a.n_rows + i];
      }
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int j = h + 2 * m;
        const int32_t src = (in && sv[m] >= 0 && (int64_t)sv[m] < a.n_rows) ? sv[m] : -1;
        if (j < K) srcs0[r * K + j] = src;
        if (j < K && src >= 0) bits |= 1u << j;
      }
      __syncthreads();  // rowmask zeroed above before any thread ORs into it
    } else {
      if (tid < BM) {
        const int64_t i = row0 + tid;
        const bool in = i < a.n_rows;
        const int2 c = reinterpret_cast<const int2*>(a.coords)[in ? i : 0];
        const bool ok = in && c.x >= 0 && c.x < a.B && c.y >= 0 && c.y < a.V;
        row_b[tid] = ok ? c.x : -1;
        row_v[tid] = ok ? c.y : -1;
      }
      __syncthreads();
      const int b = row_b[r];
      const int v = row_v[r];
      // All loads of one level are issued before any is used, unconditionally
      // (entries past K read a valid address and are masked afterwards), so the
      // whole list costs two memory round trips.
      const int vv = v >= 0 ? v : 0;
      int32_t nb[SPT];
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int j = h + 2 * m;
        nb[m] = a.nbr[(int64_t)vv * K + (j < K ? j : K - 1)];
      }
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int j = h + 2 * m;
        nb[m] = (j < K && v >= 0 && nb[m] >= 0 && nb[m] < a.V) ? nb[m] : -1;
      }
      const int bb = b >= 0 ? b : 0;
      int32_t sv[SPT];
#pragma unroll
      for (int m = 0; m < SPT; ++m) sv[m] = a.inv[(int64_t)bb * a.V + (nb[m] >= 0 ? nb[m] : 0)];
#pragma unroll
      for (int m = 0; m < SPT; ++m) {
        const int j = h + 2 * m;
        const int32_t src = (nb[m] >= 0 && sv[m] >= 0 && (int64_t)sv[m] < a.n_rows) ? sv[m] : -1;
        if (j < K) srcs0[r * K + j] = src;
        if (src >= 0) bits |= 1u << j;
      }
    }
    if (bits) atomicOr(&rowmask[r], bits);
    __syncthreads();

    // Row permutation: order the tile's rows by their first "sparse" slot
    // (a slot present in fewer than half of the rows), rows with no sparse
    // slot first and rows past the end last.  Rows sharing a sparse slot then
    // sit in the same 16-row MFMA blocks, so far fewer (block, slot) products
    // have to be computed.  Stable counting sort with wavefront ballots,
    // done by waves 0 and 1 (one row per lane).
    uint32_t rm = 0;
    int bucket = 0, rank = 0;
    if (tid < BM) {
      rm = rowmask[tid];
      const uint64_t lt = (1ull << lane) - 1ull;
      for (int j = 0; j < K; ++j) {
        const uint64_t bal = __ballot((rm >> j) & 1u);
        if (lane == 0) scnt[wave * kMaxSlots + j] = __popcll(bal);
      }
      // rows past the end and their slot counts do not matter: they are zero
      (void)lt;
    }
    __syncthreads();
    if (tid < BM) {
      uint32_t dense = 0;
      for (int j = 0; j < K; ++j)
        if (2 * (scnt[j] + scnt[kMaxSlots + j]) >= BM) dense |= 1u << j;
      const uint32_t key = rm & ~dense;
      const bool valid = row0 + tid < a.n_rows;
      bucket = !valid ? K + 1 : (key ? 1 + __builtin_ctz(key) : 0);
      const uint64_t lt = (1ull << lane) - 1ull;
      for (int bk = 0; bk <= K + 1; ++bk) {
        const uint64_t bal = __ballot(bucket == bk);
        if (bucket == bk) rank = __popcll(bal & lt);
        if (lane == 0) bcnt[wave * kBuckets + bk] = __popcll(bal);
      }
    }
    __syncthreads();
    if (tid < BM) {
      int pos = rank + (wave == 1 ? bcnt[bucket] : 0);
      for (int bk = 0; bk < bucket; ++bk) pos += bcnt[bk] + bcnt[kBuckets + bk];
      perm[pos] = tid;
    }
    __syncthreads();
    for (int e = tid; e < BM * K; e += kThreads) {
      const int p = e / K;
      const int j = e - p * K;
      srcs[e] = srcs0[perm[p] * K + j];
    }
    if (tid < BM) {
      const uint32_t m = rowmask[perm[tid]];
      if (m) atomicOr(&blk_slots[tid >> 4], m);
    }
  } else {
    __syncthreads();
    if (tid < BM) {
      const int64_t i = row0 + tid;
      const bool in = i < a.n_rows;
      int32_t src = in ? (int32_t)i : -1;
      if (a.gather) {  // input row b_i * V + v_i of the dense tensor
        const int2 c = reinterpret_cast<const int2*>(a.coords)[in ? i : 0];
        const bool ok = in && c.x >= 0 && c.x < a.B && c.y >= 0 && c.y < a.V;
        src = ok ? c.x * a.V + c.y : -1;
      }
      srcs[tid] = src;
      perm[tid] = tid;
      if (in) atomicOr(&blk_slots[tid >> 4], 1u);
    }
  }
  __syncthreads();
  uint32_t tile_slots = 0;
#pragma unroll
  for (int q = 0; q < kRowBlocks; ++q) tile_slots |= blk_slots[q];
  tile_slots = __builtin_amdgcn_readfirstlane(tile_slots);
  uint32_t my_blk[4];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
    my_blk[rb] = __builtin_amdgcn_readfirstlane(blk_slots[wm * 4 + rb]);

  // ---- reduction walk ----------------------------------------------------------
  // Slot of reduction entry kk: kk / Cin by multiply-high with the host's
  // reciprocal ceil(2^32 / Cin) (exact for kk * Cin < 2^32), no division.
  const uint32_t magic = a.cin_magic;
  auto slot_of = [&](int kk) -> int { return (int)__umulhi((uint32_t)kk, magic); };
  // slots touched by reduction entries [k_lo, k_hi), 0 past the end
  auto range_bits = [&](int k_lo, int k_hi) -> uint32_t {
    if (k_lo >= Ktot) return 0u;
    return slot_range_bits(slot_of(k_lo), slot_of(min(k_hi, Ktot) - 1));
  };

  // ---- global -> register -> LDS staging -------------------------------------
  // Every global load is issued unconditionally: an absent neighbour row or an
  // out-of-range entry reads a valid address (the first row of S or of W) and
  // the value is replaced by zero when it is written to LDS.  (Loads under a
  // divergent branch would make the compiler wait for all outstanding loads
  // and serialise the prefetch pipeline.)
  struct Regs {
    i32x4 a[Lt::AVecs];
    i32x4 w[Lt::WVecs];
    uint32_t a_ok;  // bit u: a[u] holds data (else zeros are stored)
    uint32_t w_ok;
  };

  auto load_chunk = [&](int chunk, Regs& R) {
    const int k0 = chunk * KC;
    R.a_ok = 0;
#pragma unroll
    for (int u = 0; u < Lt::AVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int r = idx / Lt::AVecPerRow;
      const int q = idx % Lt::AVecPerRow;
      const int kk = k0 + q * E::per_vec;
      const int j = CONV ? slot_of(kk) : 0;
      const int c = kk - j * Cin;
      const int32_t src = srcs[r * K + (j < K ? j : K - 1)];
      const bool ok = kk < Ktot && src >= 0;
      const int64_t off = ok ? ((int64_t)src * Cin + c) * E::bytes : 0;
      R.a[u] = *reinterpret_cast<const i32x4*>(S + off);
      R.a_ok |= ok ? (1u << u) : 0u;
    }
    R.w_ok = 0;
#pragma unroll
    for (int u = 0; u < Lt::WVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int kr = idx / Lt::WVecPerRow;
      const int q = idx % Lt::WVecPerRow;
      const int kk = k0 + kr;
      const int n = n0 + q * E::per_vec;
      const bool ok = kr < KC && kk < Ktot && n < Cout;
      const int64_t off = ok ? ((int64_t)kk * Cout + n) * E::bytes : 0;
      R.w[u] = *reinterpret_cast<const i32x4*>(W + off);
      R.w_ok |= ok ? (1u << u) : 0u;
    }
  };

  auto store_chunk = [&](const Regs& R, int buf) {
    unsigned char* a_lds = smem + buf * Lt::Stage;
    unsigned char* w_lds = a_lds + Lt::AStage;
    const i32x4 zero = {0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < Lt::AVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int r = idx / Lt::AVecPerRow;
      const int q = idx % Lt::AVecPerRow;
      *reinterpret_cast<i32x4*>(a_lds + r * Lt::ARow + q * 16) =
          ((R.a_ok >> u) & 1u) ? R.a[u] : zero;
    }
#pragma unroll
    for (int u = 0; u < Lt::WVecs; ++u) {
      const int idx = tid + u * kThreads;
      const int kr = idx / Lt::WVecPerRow;
      const int q = idx % Lt::WVecPerRow;
      if (kr < KC)
        *reinterpret_cast<i32x4*>(w_lds + kr * Lt::WRow + q * 16) =
            ((R.w_ok >> u) & 1u) ? R.w[u] : zero;
    }
  };

  // bias of this lane's columns: the accumulators start at it
  float bias_v[NB];
#pragma unroll
  for (int cb = 0; cb < NB; ++cb) {
    const int col = n0 + wn * WN + cb * 16 + l16;
    const bool ok = a.bias != nullptr && col < Cout;
    const float* bp = a.bias != nullptr ? a.bias : reinterpret_cast<const float*>(a.W);
    const float bvl = bp[ok ? col : 0];
    bias_v[cb] = ok ? bvl : 0.f;
  }
  f32x4 acc[4][NB];
#pragma unroll
  for (int rb = 0; rb < 4; ++rb)
#pragma unroll
    for (int cb = 0; cb < NB; ++cb)
      acc[rb][cb] = f32x4{bias_v[cb], bias_v[cb], bias_v[cb], bias_v[cb]};

  // one 64-byte k-step (32 bf16 / 16 fp32 reduction entries) of a staged chunk
  auto compute_step = [&](const unsigned char* a_lds, const unsigned char* w_lds, int ks,
                          uint32_t bits) {
    if (BF16) {
      bf16x8 bfrag[NB];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        // k rows 8g + (0..3 | 4..7) of the step, columns cb*16 + 4*(l16 % 4) + 0..3
        const int col = wn * WN + cb * 16 + 4 * (l16 & 3);
        const int kr = ks * 32 + 8 * g + (l16 >> 2);
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
        const i32x4 af =
            *reinterpret_cast<const i32x4*>(a_lds + row * Lt::ARow + ks * 64 + g * 16);
        const bf16x8 afrag = __builtin_bit_cast(bf16x8, af);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
          acc[rb][cb] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(afrag, bfrag[cb], acc[rb][cb], 0, 0, 0);
      }
    } else {
      // fp32: lane group g holds k = 4g .. 4g+3 of the step's 16 entries;
      // MFMA s uses component s of the A vector and W row 4g + s.
      float bw[NB][4];
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const int col = wn * WN + cb * 16 + l16;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2)
          bw[cb][s2] = *reinterpret_cast<const float*>(
              w_lds + (ks * 16 + 4 * g + s2) * Lt::WRow + col * 4);
      }
#pragma unroll
      for (int rb = 0; rb < 4; ++rb) {
        if ((my_blk[rb] & bits) == 0u) continue;
        const int row = wm * 64 + rb * 16 + l16;
        const i32x4 af =
            *reinterpret_cast<const i32x4*>(a_lds + row * Lt::ARow + ks * 64 + g * 16);
#pragma unroll
        for (int cb = 0; cb < NB; ++cb)
#pragma unroll
          for (int s2 = 0; s2 < 4; ++s2)
            acc[rb][cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                __int_as_float(af[s2]), bw[cb][s2], acc[rb][cb], 0, 0, 0);
      }
    }
  };

  auto compute = [&](int chunk, int buf) {
    const unsigned char* a_lds = smem + buf * Lt::Stage;
    const unsigned char* w_lds = a_lds + Lt::AStage;
    constexpr int KS = KC / Lt::KSTEP;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const int klo = chunk * KC + ks * Lt::KSTEP;
      const uint32_t bits = __builtin_amdgcn_readfirstlane(range_bits(klo, klo + Lt::KSTEP));
      compute_step(a_lds, w_lds, ks, bits);
    }
  };

  // ---- main loop -------------------------------------------------------------

  // ---- main loop: software pipeline over steps t = 0, 1, ... ---------------------
  // Step t loads chunk t into register set t % 2, runs the MFMAs of chunk
  // t - 2 from LDS buffer t % 2, and stores chunk t - 1 (register set
  // (t - 1) % 2, loaded one step earlier) into LDS buffer (t - 1) % 2; one
  // barrier per step.  A chunk's loads thus have two steps of MFMA work to
  // arrive.  Every step issues its loads (past the end they re-read the last
  // chunk): a load under even a uniform branch leaves the compiler unsure how
  // many loads are outstanding, and it then waits for all of them.  The trip
  // count is even so the two register sets keep fixed roles.
  if (STAGES == 2) {
    const int last = nchunks - 1;
    const int nsteps = (nchunks + 3) & ~1;  // >= nchunks + 2, even
    Regs R0, R1;
    for (int t = 0; t < nsteps; t += 2) {
      // even step t: buffers t % 2 = 0 (compute) and 1 (store)
      load_chunk(min(t, last), R0);
      if (t >= 2) compute(t - 2, 0);
      if (t >= 1 && t - 1 < nchunks) store_chunk(R1, 1);
      __syncthreads();
      // odd step t + 1
      load_chunk(min(t + 1, last), R1);
      if (t + 1 >= 2 && t - 1 < nchunks) compute(t - 1, 1);
      if (t < nchunks) store_chunk(R0, 0);
      __syncthreads();
    }
  } else {
    // single LDS buffer: loads run one chunk ahead in registers; two barriers per chunk
    const int last = nchunks - 1;
    Regs R;
    load_chunk(0, R);
    store_chunk(R, 0);
    __syncthreads();
    for (int c = 0; c < nchunks; ++c) {
      load_chunk(min(c + 1, last), R);
      compute(c, 0);
      __syncthreads();
      if (c + 1 < nchunks) {
        store_chunk(R, 0);
        __syncthreads();
      }
    }
  }

  // ---- epilogue: bias + activation + rounding, staged through LDS -----------
  // LDS row p holds tile row perm[p]; rows are written back as 16-byte vectors.
  unsigned char* o_lds = smem;
  unsigned char* out = static_cast<unsigned char*>(a.out);
  constexpr int kVecPerRow = BN * E::bytes / 16;
  constexpr int kPasses = Lt::OnePassOut ? 1 : 2;
  constexpr int kRowsPerPass = BM / kPasses;
  const int ncols = min(BN, Cout - n0);
  const int vec_valid = ncols * E::bytes / 16;
  for (int pass = 0; pass < kPasses; ++pass) {
    if (kPasses == 1 || wm == pass) {
#pragma unroll
      for (int cb = 0; cb < NB; ++cb) {
        const int col_l = wn * WN + cb * 16 + l16;
#pragma unroll
        for (int rb = 0; rb < 4; ++rb) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int row_l = (kPasses == 1 ? wm * 64 : 0) + rb * 16 + g * 4 + r;
            float v = acc[rb][cb][r];  // the bias is already in
            if (a.relu) v = v > 0.f ? v : 0.f;
            unsigned char* p = o_lds + row_l * Lt::ORow + col_l * E::bytes;
            if (BF16)  // hardware round-to-nearest-even conversion
              *reinterpret_cast<__bf16*>(p) = static_cast<__bf16>(v);
            else
              *reinterpret_cast<float*>(p) = v;
          }
        }
      }
    }
    __syncthreads();
    for (int idx = tid; idx < kRowsPerPass * kVecPerRow; idx += kThreads) {
      const int r = idx / kVecPerRow;
      const int q = idx % kVecPerRow;
      const int64_t i = row0 + perm[pass * kRowsPerPass + r];
      if (i < a.n_rows && q < vec_valid) {
        const i32x4 v = *reinterpret_cast<const i32x4*>(o_lds + r * Lt::ORow + q * 16);
        *reinterpret_cast<i32x4*>(out + (i * Cout + n0) * E::bytes + q * 16) = v;
      }
    }
    if (kPasses == 2) __syncthreads();
  }
}

template <typename Kern>
hipError_t launch_kernel(Kern kern, unsigned gx, unsigned gy, size_t lds, hipStream_t stream,
                         const GemmArgs& a) {
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

#ifndef SHC_GEMM_CHUNK
#define SHC_GEMM_CHUNK 64
#endif
#ifndef SHC_GEMM_STAGES
#define SHC_GEMM_STAGES 2
#endif

template <bool BF16, int BN, bool CONV>
hipError_t launch_tile(const GemmArgs& a_in, hipStream_t stream) {
  constexpr int CH = SHC_GEMM_CHUNK;
  constexpr int ST = SHC_GEMM_STAGES;
  GemmArgs a = a_in;
  a.cin_magic = (uint32_t)(((1ull << 32) + (uint64_t)a.Cin - 1) / (uint64_t)a.Cin);
  const unsigned gx = (unsigned)((a.n_rows + BM - 1) / BM);
  const unsigned gy = (unsigned)((a.Cout + BN - 1) / BN);
  const size_t lds = lds_bytes<BF16, BN, CH, ST>(CONV ? a.K : 1);
  if (!CONV)
    return launch_kernel(gather_gemm_kernel<BF16, BN, false, false, CH, ST, 1>, gx, gy, lds,
                         stream, a);
  if (a.table != nullptr) {
    if (a.K <= 10)
      return launch_kernel(gather_gemm_kernel<BF16, BN, true, true, CH, ST, 5>, gx, gy, lds,
                           stream, a);
    return launch_kernel(gather_gemm_kernel<BF16, BN, true, true, CH, ST, kMaxSlots / 2>, gx,
                         gy, lds, stream, a);
  }
  if (a.K <= 10)
    return launch_kernel(gather_gemm_kernel<BF16, BN, true, false, CH, ST, 5>, gx, gy, lds,
                         stream, a);
  return launch_kernel(gather_gemm_kernel<BF16, BN, true, false, CH, ST, kMaxSlots / 2>, gx, gy,
                       lds, stream, a);
}

template <bool BF16, bool CONV>
hipError_t launch_typed(const GemmArgs& a, hipStream_t stream) {
  if (a.Cout >= 128) return launch_tile<BF16, 128, CONV>(a, stream);
  return launch_tile<BF16, 64, CONV>(a, stream);
}

}  // namespace

hipError_t launch_gather_gemm(const GemmArgs& a, bool conv, bool bf16, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  // weight-stationary kernel when a column slice of W fits in LDS
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  // The slot-major conv (every output column per workgroup, the slots in
  // turn) against the weight-stationary one (column slices of W resident,
  // jobs of 16 rows x slot), measured at K = 9 (the same results bit for
  // bit): faster from about 1000 rows per CU (the density-sweep batch at
  // 20 / 50 / 100%: 112 / 282 / 612 us against 138 / 347 / 659 us; the
  // full-mesh cap at 64 channels 54 against 95 us) and for 64 input
  // channels within one round of 128-row groups (6.6 against 10.6 us at
  // 4,200 rows); slower for 128 input channels at a few hundred rows per CU
  // (36 against 26 us at 5% of the density-sweep batch).
  if (conv && conv_sm_supported(a, bf16) &&
      (a.n_rows >= 1000LL * cus || (a.Cin == 64 && a.n_rows <= 128LL * cus)))
    return launch_conv_sm(a, cus, stream);
  WsPlan plan;
  if (ws_plan(a, conv, bf16, cus, &plan)) return launch_ws_gemm(a, conv, bf16, plan, stream);
  // a conv plan exists only for the weight-stationary kernel
  if (a.plan != nullptr || a.plan_out != nullptr) return hipErrorInvalidValue;
  if (bf16) return conv ? launch_typed<true, true>(a, stream) : launch_typed<true, false>(a, stream);
  return conv ? launch_typed<false, true>(a, stream) : launch_typed<false, false>(a, stream);
}

}  // namespace shc
