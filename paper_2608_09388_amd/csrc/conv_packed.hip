// Sparse neighbourhood convolution from a neighbour-row table (Eqs. 4-5,
// with the activation of Eq. 10), bf16, with every slot's weights held in
// registers for the whole launch:
//
//   out[i] = act( bias + sum_{j < K, table[j][i] present} S[table[j][i]] W[j] ).
//
// The weights come pre-arranged (shc_pack_conv_weights): for slot j, output
// column block ct (16 columns) and k-step ks (32 input channels), the 64
// lanes' A-operand fragments of a 16x16x32 bf16 MFMA lie in 1 KB, so each
// wavefront loads its fragments with plain 16-byte loads, straight into
// registers, with no LDS transpose.
//
// One workgroup per CU of one wavefront per 16 output columns (eight for
// 128 columns: two per SIMD); a wavefront holds the fragments of every slot
// for its columns (for 128 -> 128 and K = 9: 144 registers a lane).  A
// workgroup takes a chunk of consecutive active rows (about N' / CUs, so one
// round of workgroups covers the rows) and
//   1. loads slot 0's fragments and the chunk's table entries into
//      registers (the other slots' fragments follow while it groups);
//   2. groups the rows in LDS by two keys, whether any present neighbour lies
//      outside the chunk, then the first present slot after slot 0 (one LDS
//      counter per key; the order within a key is immaterial), so that a
//      16-row block mostly shares its slots;
//   3. writes every (position, slot) entry as the LDS row its operand is
//      read from: a neighbour in the chunk from the chunk's copy, the others
//      from staging rows filled in rounds of at most PCAP rows, an absent
//      one from a row of zeros;
//   4. loads the chunk's rows into LDS in position order and the round's
//      staged rows (direct global->LDS loads, 16-byte chunks swizzled by
//      row), then multiplies, block by block, every slot present in any of
//      the block's rows, slot 0 first and the others ascending, into one
//      fp32 accumulator.
// Steps 1-3 depend only on the table: the plan launch runs them alone and
// writes each chunk's result out (an image of the LDS it filled), and the
// planned conv reads that image back in their place.
// Each row's sum runs in a fixed order (slots ascending, each MFMA's 32
// products as the hardware sums them), so the result does not depend on the
// grid or on where a row lands in the sort.  Then bias, activation and the
// rounding to bf16, stored straight from the accumulators.
//
// MFMAs run transposed (D^T = W^T S^T): lane (g, i) of a 16 x 16 result holds
// output columns 4g .. 4g+3 of the block's row i.
#include <hip/hip_runtime.h>

#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kPkMaxK = 9;                  // slots held in registers
constexpr int kPkKeys = 2 * kPkMaxK;        // sort keys: (staged?, first slot after 0)
constexpr int kPkLdsLimit = 160 * 1024;
#define SHC_PK_LDS __attribute__((address_space(3)))

typedef __bf16 pk_bf16x2 __attribute__((ext_vector_type(2)));
typedef float pk_f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t pk_v2u32 __attribute__((ext_vector_type(2)));
typedef uint32_t pk_v4u32 __attribute__((ext_vector_type(4)));

struct PackedArgs {
  const void* S;          // [n_rows][Cin] bf16
  const int32_t* table;   // [K][n_rows]
  const void* Wp;         // packed weights, [K][Cout/16][Cin/32][64 lanes][8] bf16
  const float* bias;      // [Cout] or null
  void* out;              // [n_rows][Cout] bf16
  int64_t n_rows;
  int32_t K;
  int32_t relu;
  int32_t chunk_rows;     // rows per chunk (<= RMAX)
  int32_t n_chunks;
  void* plan;             // chunk images (plan launch: written; planned conv: read)
};

// The three launches of one kernel body: the conv grouping its rows itself,
// the plan (the grouping alone, written out per chunk), and the conv reading
// a plan.
enum PkMode { kPkFull = 0, kPkPlan = 1, kPkPlanned = 2 };

// Per shape: wavefronts (one 16-column block each), rows of the chunk held
// in LDS, staged neighbour rows per round, and the LDS layout (bytes).
template <int KS, int NCT>
struct PkShape {
  static constexpr int NW = NCT;
  static constexpr int NT = 64 * NW;
  static constexpr int Cin = KS * 32;
  static constexpr int RB = Cin * 2;        // bytes of a row
  static constexpr int VPR = RB / 16;       // 16-byte chunks of a row
  static constexpr int RMAX = KS >= 4 ? 320 : 512;
  static constexpr int PCAP = KS >= 4 ? 192 : 384;
  static constexpr int RPT = (RMAX + NT - 1) / NT;  // rows per thread
  static constexpr int NPOS = RPT * NT;             // positions a scan covers
  static constexpr int SMAX = RMAX * kPkMaxK;       // staged pairs of a chunk, at most
  static constexpr int ZROW = RMAX + PCAP;                      // a row of zeros
  static constexpr int NBLK = RMAX / 16;                         // 16-row blocks of a chunk
  // the chunk's plan: what the blocks read, in one contiguous image (the
  // packed-plan launch writes it to global memory, the planned conv reads
  // it back): positions' rows, slot entries, block slot sets, rounds, block
  // boundaries in the staging list, header, staging sources
  static constexpr int off_prow = (ZROW + 1) * RB;               // uint16 [RMAX]
  static constexpr int off_ltab = off_prow + RMAX * 2;           // uint16 [RMAX][16]
  static constexpr int off_union = off_ltab + RMAX * 32;         // uint32 [NBLK]
  static constexpr int off_rnd = off_union + NBLK * 4;           // int32 [NBLK + 2]
  static constexpr int off_bnd = off_rnd + (NBLK + 2) * 4;       // int32 [NBLK + 1]
  static constexpr int off_hdr = off_bnd + (NBLK + 1) * 4;       // int32 [4]
  static constexpr int off_ssrc = (off_hdr + 16 + 15) / 16 * 16;  // int32 [SMAX]
  static constexpr int IMG = (off_ssrc + SMAX * 4 + 15) / 16 * 16 - off_prow;
  // working arrays of the grouping
  static constexpr int off_rowpos = off_prow + IMG;              // uint16 [RMAX]
  static constexpr int off_obase = off_rowpos + RMAX * 2;        // int32 [NPOS + 1]
  static constexpr int off_hist = off_obase + (NPOS + 1) * 4;    // int32 [kPkKeys]
  static constexpr int off_kbase = off_hist + kPkKeys * 4;       // int32 [kPkKeys + 1]
  static constexpr int off_wsum = off_kbase + (kPkKeys + 1) * 4;  // int32 [NW]
  static constexpr int off_bsb = off_wsum + NW * 4;              // int32 [NBLK]
  static constexpr int bytes = off_bsb + NBLK * 4;
  static_assert(off_ltab % 16 == 0 && off_prow % 16 == 0, "aligned slot entries");
  static_assert(bytes <= kPkLdsLimit, "one workgroup per CU");
  static_assert(RMAX % 16 == 0 && PCAP >= 16 * kPkMaxK, "chunk shape");
  static_assert(ZROW < 65536, "LDS rows fit 16 bits");
  static_assert(NBLK + 1 <= 64, "one wavefront holds the block boundaries");
  static_assert(kPkKeys <= 64, "one wavefront scans the keys");
};

// A workgroup barrier that orders LDS only (global loads stay in flight).
__device__ __forceinline__ void pk_lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// inclusive prefix sum over the wavefront's lanes
__device__ __forceinline__ int pk_wave_scan(int v, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int t = __shfl_up(v, d);
    if (lane >= d) v += t;
  }
  return v;
}

// Workgroup b's first chunk: workgroups are dealt to the eight XCDs in turn,
// so consecutive chunks (whose rows' neighbours overlap) go to one XCD's L2.
__device__ __forceinline__ int pk_first_chunk(int b, int grid) {
  const int x = b & 7, i = b >> 3, q = grid >> 3, r = grid & 7;
  return x * q + (x < r ? x : r) + i;
}

// LDS byte offset of 16-byte chunk c of LDS row L (chunk swizzled by row)
template <int VPR, int RB>
__device__ __forceinline__ int pk_chunk_at(int L, int c) {
  return L * RB + ((c ^ (L & (VPR - 1))) << 4);
}

template <int KS, int NCT, int MODE>
__global__ __launch_bounds__(64 * NCT, 1) void conv_packed_kernel(const PackedArgs a) {
  using SH = PkShape<KS, NCT>;
  constexpr int NT = SH::NT, RPT = SH::RPT;
  constexpr int Cout = NCT * 16;
  constexpr int RB = SH::RB, VPR = SH::VPR, RMAX = SH::RMAX, PCAP = SH::PCAP;

  extern __shared__ __attribute__((aligned(16))) unsigned char smem_base[];
  // the plan launch holds no rows: its LDS starts at the plan image
  unsigned char* smem = MODE == kPkPlan ? smem_base - SH::off_prow : smem_base;
  unsigned char* rows = smem;  // [RMAX] chunk rows, then [PCAP] staged rows
  uint16_t* prow = reinterpret_cast<uint16_t*>(smem + SH::off_prow);      // position -> row
  uint16_t* rowpos = reinterpret_cast<uint16_t*>(smem + SH::off_rowpos);  // row -> position
  int32_t* obase = reinterpret_cast<int32_t*>(smem + SH::off_obase);
  uint16_t* ltab = reinterpret_cast<uint16_t*>(smem + SH::off_ltab);
  int32_t* ssrc = reinterpret_cast<int32_t*>(smem + SH::off_ssrc);
  int32_t* hist = reinterpret_cast<int32_t*>(smem + SH::off_hist);
  int32_t* kbase = reinterpret_cast<int32_t*>(smem + SH::off_kbase);
  uint32_t* bunion = reinterpret_cast<uint32_t*>(smem + SH::off_union);
  int32_t* wsum = reinterpret_cast<int32_t*>(smem + SH::off_wsum);
  int32_t* blk_sb = reinterpret_cast<int32_t*>(smem + SH::off_bsb);
  int32_t* rnd = reinterpret_cast<int32_t*>(smem + SH::off_rnd);
  int32_t* bnd = reinterpret_cast<int32_t*>(smem + SH::off_bnd);
  int32_t* hdr = reinterpret_cast<int32_t*>(smem + SH::off_hdr);
  constexpr int ZROW = SH::ZROW, NBLK = SH::NBLK, IMG = SH::IMG;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;  // owns output columns 16 wave .. 16 wave + 15
  const int g = lane >> 4;
  const int l16 = lane & 15;
  const int64_t n = a.n_rows;
  const int K = a.K;
  const unsigned char* S = static_cast<const unsigned char*>(a.S);

  // every slot's weight fragments of this wavefront's columns, for good
  // (slots from K on read the buffer out of range, as zeros, and are never
  // used: no row has them)
  bf16x8 wreg[kPkMaxK][KS];
  const __amdgpu_buffer_rsrc_t w_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.Wp), (short)0, K * KS * NCT * 1024, 0x00020000);
  const uint32_t w_lane = (uint32_t)(lane * 16 + wave * KS * 1024);
  auto load_w = [&](int j0, int j1) {
#pragma unroll
    for (int j = 0; j < kPkMaxK; ++j)
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        if (j >= j0 && j < j1)
          wreg[j][ks] = __builtin_bit_cast(
              bf16x8, __builtin_amdgcn_raw_buffer_load_b128(w_rsrc, w_lane,
                                                            (j * NCT * KS + ks) * 1024, 0));
  };
  // slot 0's fragments now; the other slots' after the first chunk's table
  // entries, so that the grouping waits for slot 0's and the table only (a
  // planned conv loads them all beside its first chunk's plan; the plan
  // launch needs none)
  if (MODE == kPkFull) load_w(0, 1);
  if (MODE == kPkPlanned) load_w(0, kPkMaxK);
  bool w_rest = MODE == kPkFull;
  f32x4 bias4;
  {
    const int col = wave * 16 + 4 * g;
    bias4 = a.bias ? f32x4{a.bias[col], a.bias[col + 1], a.bias[col + 2], a.bias[col + 3]}
                   : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  // the row of zeros that absent neighbours read (published by the chunk's
  // first barrier)
  if (MODE != kPkPlan && tid < VPR)
    *reinterpret_cast<pk_v4u32*>(rows + ZROW * RB + tid * 16) = pk_v4u32{0, 0, 0, 0};
  // lane constant of the B-operand addresses: 16-byte chunk 4 ks + g of a row
  int gk[KS];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) gk[ks] = (ks * 4 + g) << 4;
  const __amdgpu_buffer_rsrc_t t_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<int32_t*>(a.table), (short)0, (int)(K * n * 4), 0x00020000);

  for (int64_t chunk = pk_first_chunk(blockIdx.x, gridDim.x); chunk < a.n_chunks;
       chunk += gridDim.x) {
    const int64_t row0 = chunk * a.chunk_rows;
    const int nrows = (int)min((int64_t)a.chunk_rows, n - row0);
    const int nblk = (nrows + 15) >> 4;
    int nin;
    if constexpr (MODE == kPkPlanned) {
      // the chunk's plan image into LDS (direct loads), then its header: a
      // plan of another row count or chunking is refused chunk by chunk
      const unsigned char* img = static_cast<const unsigned char*>(a.plan) + chunk * (int64_t)IMG;
      for (int v0 = wave * 64; v0 < IMG / 16; v0 += NT) {
        const int v = v0 + lane;
        if (v < IMG / 16)
          __builtin_amdgcn_global_load_lds(img + v * 16,
                                           (SHC_PK_LDS void*)(smem + SH::off_prow + v0 * 16), 16,
                                           0, 0);
      }
      __builtin_amdgcn_s_waitcnt(0);
      pk_lds_barrier();
      if (hdr[1] != nrows || hdr[2] != (int)(n & 0x7FFFFFFF) || hdr[3] != (int)chunk) {
        pk_lds_barrier();
        continue;
      }
      nin = hdr[0];
    } else {
    // 1. the table entries of this thread's rows (branch-free: an entry past
    // the chunk or the slots reads the buffer out of range); the key counts
    // and block unions start at zero
    int32_t tv[RPT][kPkMaxK];
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int t = u * NT + tid;
#pragma unroll
      for (int j = 0; j < kPkMaxK; ++j) {
        const bool in = t < nrows && j < K;
        const uint32_t off = (uint32_t)(((int64_t)j * n + row0 + t) * 4);
        const int32_t e = (int32_t)__builtin_amdgcn_raw_buffer_load_b32(
            t_rsrc, in ? off : 0x80000000u, 0, 0);
        tv[u][j] = in ? e : -1;
      }
    }
    if (w_rest) {
      load_w(1, kPkMaxK);
      w_rest = false;
    }
    if (tid < kPkKeys) hist[tid] = 0;
    if (tid < RMAX / 16) bunion[tid] = 0u;
    pk_lds_barrier();

    // 2. keys (any staged neighbour, then the first present slot after slot
    // 0) and each row's rank among its key's rows; the order within a key is
    // immaterial, so one LDS atomic per row gives it
    uint32_t m[RPT];
    int key[RPT], rank[RPT], nst[RPT];
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      const int t = u * NT + tid;
      uint32_t mm = 0;
      int staged = 0;
#pragma unroll
      for (int j = 0; j < kPkMaxK; ++j) {
        const bool present = (uint64_t)(uint32_t)tv[u][j] < (uint64_t)n;
        mm |= (uint32_t)present << j;
        staged += (int)(present && (uint64_t)(tv[u][j] - row0) >= (uint64_t)nrows);
      }
      m[u] = mm;
      nst[u] = staged;
      const uint32_t rest = mm & ~1u;
      key[u] = t < nrows ? (staged > 0) * kPkMaxK + (rest ? (int)__builtin_ctz(rest) : 0) : -1;
      rank[u] = key[u] >= 0 ? atomicAdd(&hist[key[u]], 1) : 0;
    }
    pk_lds_barrier();
    if (wave == 0) {
      const int h = lane < kPkKeys ? hist[lane] : 0;
      const int incl = pk_wave_scan(h, lane);
      if (lane < kPkKeys) kbase[lane] = incl - h;
      if (lane == kPkKeys - 1) kbase[kPkKeys] = incl;
    }
    pk_lds_barrier();
    // 3. positions; rows with no staged neighbour come first (nin of them)
    int pos[RPT];
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      pos[u] = -1;
      if (key[u] >= 0) {
        pos[u] = kbase[key[u]] + rank[u];
        prow[pos[u]] = (uint16_t)(u * NT + tid);
        rowpos[u * NT + tid] = (uint16_t)pos[u];
        obase[pos[u]] = nst[u];
        atomicOr(&bunion[pos[u] >> 4], m[u]);
      }
    }
    nin = kbase[kPkMaxK];
    pk_lds_barrier();
    // 4. staged-pair numbers by position (exclusive prefix over positions)
    {
      int c[RPT], sum = 0;
#pragma unroll
      for (int e = 0; e < RPT; ++e) {
        const int p = tid * RPT + e;
        c[e] = p < nrows ? obase[p] : 0;
        sum += c[e];
      }
      const int incl = pk_wave_scan(sum, lane);
      if (lane == 63) wsum[wave] = incl;
      pk_lds_barrier();
      int run = incl - sum;
      for (int w = 0; w < wave; ++w) run += wsum[w];
#pragma unroll
      for (int e = 0; e < RPT; ++e) {
        obase[tid * RPT + e] = run;
        run += c[e];
      }
      if (tid == NT - 1) obase[SH::NPOS] = run;
    }
    pk_lds_barrier();
    // rounds: blocks from nin / 16 on (those holding staged rows) in runs
    // whose staged rows fit the PCAP staging rows; blk_sb[b] is the first
    // staging-list entry of block b's round, rnd[] the rounds' first blocks
    // (then nblk), rnd[NBLK + 1] their count
    if (wave == 0) {
      const int bs0 = nin >> 4;
      const int nsb = nblk - bs0;
      const int bt = lane <= nsb ? obase[min((bs0 + lane) * 16, nrows)] : 0;
      int sb = 0, nr = 0;
      for (int t = 0; t < nsb; ++t) {
        if (t == 0 || __builtin_amdgcn_readlane(bt, t + 1) - sb > PCAP) {
          sb = __builtin_amdgcn_readlane(bt, t);
          if (lane == 0) rnd[nr] = bs0 + t;
          ++nr;
        }
        if (lane == 0) blk_sb[bs0 + t] = sb;
      }
      if (lane == 0) {
        rnd[nr] = nblk;
        rnd[NBLK + 1] = nr;
      }
    }
    pk_lds_barrier();
    // 5. each row's slot entries at its position, as LDS rows: an in-chunk
    // neighbour's position, a staged one's row in its round's staging rows,
    // ZROW for none (also for the positions past the chunk in its last block)
#pragma unroll
    for (int u = 0; u < RPT; ++u) {
      if (pos[u] >= 0) {
        int si = obase[pos[u]];
        const int base = RMAX - blk_sb[pos[u] >> 4];
        uint16_t* lt = ltab + pos[u] * 16;
#pragma unroll
        for (int j = 0; j < kPkMaxK; ++j) {
          int e = ZROW;
          if ((m[u] >> j) & 1) {
            const int64_t off = tv[u][j] - row0;
            if ((uint64_t)off < (uint64_t)nrows) {
              e = rowpos[off];
            } else {
              e = base + si;
              ssrc[si] = tv[u][j];
              ++si;
            }
          }
          lt[j] = (uint16_t)e;
        }
      }
      const int q = u * NT + tid;
      if (q >= nrows && q < nblk * 16) {
#pragma unroll
        for (int j = 0; j < kPkMaxK; ++j) ltab[q * 16 + j] = (uint16_t)ZROW;
      }
    }
    // block boundaries in the staging list, and the header
    if (tid <= nblk) bnd[tid] = obase[min(tid * 16, nrows)];
    if (tid == 0) {
      hdr[0] = nin;
      hdr[1] = nrows;
      hdr[2] = (int)(n & 0x7FFFFFFF);
      hdr[3] = (int)chunk;
    }
    pk_lds_barrier();
    if constexpr (MODE == kPkPlan) {
      // the chunk's image out, then the next chunk
      unsigned char* img = static_cast<unsigned char*>(a.plan) + chunk * (int64_t)IMG;
      for (int v = tid; v < IMG / 16; v += NT)
        *reinterpret_cast<pk_v4u32*>(img + v * 16) =
            *reinterpret_cast<const pk_v4u32*>(smem + SH::off_prow + v * 16);
      pk_lds_barrier();
      continue;
    }
    }  // steps 1-5

    // 6. blocks [b0, b1): every lane reads an operand for every slot present
    // in the block (a row without the slot reads the row of zeros)
    auto compute = [&](int b0, int b1) {
      if (b0 >= b1) return;
      // the next block's slot entries and slot set are read while a block
      // computes
      int p = b0 * 16 + l16;
      pk_v4u32 lt0 = *reinterpret_cast<const pk_v4u32*>(ltab + p * 16);
      uint32_t lt8 = *reinterpret_cast<const uint32_t*>(ltab + p * 16 + 8);
      uint32_t un = bunion[b0];
      for (int b = b0; b < b1; ++b) {
        const int pn = (b + 1 < b1 ? b + 1 : b) * 16 + l16;
        const pk_v4u32 nlt0 = *reinterpret_cast<const pk_v4u32*>(ltab + pn * 16);
        const uint32_t nlt8 = *reinterpret_cast<const uint32_t*>(ltab + pn * 16 + 8);
        const uint32_t nun = bunion[pn >> 4];
        f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int j = 0; j < kPkMaxK; ++j) {
          if (!((un >> j) & 1)) continue;
          const uint32_t word = j < 8 ? lt0[j >> 1] : lt8;
          const int L = (int)((word >> (16 * (j & 1))) & 0xFFFFu);
          const int rbase = L * RB;
          const int sw = (L & (VPR - 1)) << 4;
          bf16x8 bop[KS];
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            bop[ks] = *reinterpret_cast<const bf16x8*>(rows + rbase + (gk[ks] ^ sw));
#pragma unroll
          for (int ks = 0; ks < KS; ++ks)
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wreg[j][ks], bop[ks], acc, 0, 0, 0);
          // the slot's operand reads issue together, ahead of its MFMAs
          __builtin_amdgcn_sched_group_barrier(0x100, KS, 0);
          __builtin_amdgcn_sched_group_barrier(0x008, KS, 0);
        }
        const int prw = p < nrows ? prow[p] : nrows;
        if (prw < nrows) {
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float x = acc[r] + bias4[r];
            v[r] = a.relu ? (x > 0.f ? x : 0.f) : x;
          }
          const pk_bf16x2 h0 = __builtin_convertvector(pk_f32x2{v[0], v[1]}, pk_bf16x2);
          const pk_bf16x2 h1 = __builtin_convertvector(pk_f32x2{v[2], v[3]}, pk_bf16x2);
          unsigned char* orow = static_cast<unsigned char*>(a.out) +
                                (row0 + prw) * (int64_t)(Cout * 2) + wave * 32 + g * 8;
          *reinterpret_cast<pk_v2u32*>(orow) =
              pk_v2u32{__builtin_bit_cast(uint32_t, h0), __builtin_bit_cast(uint32_t, h1)};
        }
        p = pn;
        lt0 = nlt0;
        lt8 = nlt8;
        un = nun;
      }
    };

    // 7. the chunk's rows and the first round of staged rows; blocks wholly
    // inside the first nin positions need no staged row, the rest run in
    // rounds of at most PCAP staged rows
    // (in position order: a block's own rows then sit on 16 consecutive LDS
    // rows, whose swizzles differ, and its slot-0 reads are free of bank
    // conflicts)
    {
      const int nvec = nrows * VPR;
      const unsigned char* src = S + row0 * RB;
      for (int v0 = wave * 64; v0 < nvec; v0 += NT) {
        const int v = v0 + lane;
        const int L = v / VPR;
        const int c = (v % VPR) ^ (L & (VPR - 1));
        const int r = v < nvec ? prow[L] : 0;
        if (v < nvec && r < nrows)
          __builtin_amdgcn_global_load_lds(src + r * RB + c * 16,
                                           (SHC_PK_LDS void*)(rows + v0 * 16), 16, 0, 0);
      }
    }
    // (every index read from the plan is clamped to the chunk: a plan built
    // for another table of the same row count gives wrong values, never an
    // access out of range)
    nin = min(max(nin, 0), nrows);
    const int nr = min(max(rnd[NBLK + 1], 0), nblk);
    for (int r = 0; r == 0 || r < nr; ++r) {
      const int bs = nr ? min(max(rnd[r], 0), nblk) : nblk;
      const int be = nr ? min(max(rnd[r + 1], bs), nblk) : nblk;
      const int sb = min(max(bnd[bs], 0), SH::SMAX);
      const int nvec = min(max(bnd[be] - sb, 0), PCAP) * VPR;
      for (int v0 = wave * 64; v0 < nvec; v0 += NT) {
        const int v = v0 + lane;
        const int q = v / VPR;
        const int L = RMAX + q;
        const int c = (v % VPR) ^ (L & (VPR - 1));
        const int64_t src = v < nvec ? ssrc[min(sb + q, SH::SMAX - 1)] : 0;
        if (v < nvec && (uint64_t)src < (uint64_t)n)
          __builtin_amdgcn_global_load_lds(S + src * RB + c * 16,
                                           (SHC_PK_LDS void*)(rows + RMAX * RB + v0 * 16), 16, 0,
                                           0);
      }
      // each wavefront waits for its own direct loads; the barrier
      // publishes everyone's
      __builtin_amdgcn_s_waitcnt(0);
      pk_lds_barrier();
      if (r == 0) compute(0, nin >> 4);
      compute(bs, be);
      pk_lds_barrier();  // the staging rows and the lists are free again
    }
  }
}

__global__ void pack_weights_kernel(const uint16_t* W, int32_t K, int32_t Cin, int32_t Cout,
                                    uint16_t* Wp) {
  // Wp[((j * NCT + ct) * KS + ks) * 64 + lane][e] = W[j][32 ks + 8 g + e][16 ct + i],
  // lane = 16 g + i
  const int KS = Cin / 32, NCT = Cout / 16;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)K * NCT * KS * 64;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  int64_t rest = idx >> 6;
  const int ks = (int)(rest % KS);
  rest /= KS;
  const int ct = (int)(rest % NCT);
  const int j = (int)(rest / NCT);
  const int gg = lane >> 4, i = lane & 15;
  const uint16_t* src = W + ((int64_t)j * Cin + 32 * ks + 8 * gg) * Cout + 16 * ct + i;
  uint16_t v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = src[(int64_t)e * Cout];
  uint16_t* dst = Wp + idx * 8;
#pragma unroll
  for (int e = 0; e < 8; ++e) dst[e] = v[e];
}

// Rows per chunk: about one chunk per CU, at most RMAX.
template <int KS, int NCT>
void packed_chunks(int64_t n_rows, int num_cus, int32_t* rc_out, int32_t* chunks_out) {
  using SH = PkShape<KS, NCT>;
  int64_t rc = (n_rows + num_cus - 1) / num_cus;
  if (rc > SH::RMAX) rc = SH::RMAX;
  if (rc < 16) rc = 16;
  *rc_out = (int32_t)rc;
  *chunks_out = (int32_t)((n_rows + rc - 1) / rc);
}

template <int KS, int NCT, int MODE>
hipError_t launch_packed_k(const PackedArgs& a0, int num_cus, hipStream_t stream) {
  using SH = PkShape<KS, NCT>;
  PackedArgs a = a0;
  packed_chunks<KS, NCT>(a.n_rows, num_cus, &a.chunk_rows, &a.n_chunks);
  // the conv: one workgroup per CU; the plan launch (LDS for the plan image
  // only) every chunk at once
  const int grid = MODE == kPkPlan || a.n_chunks < num_cus ? a.n_chunks : num_cus;
  const int lds = MODE == kPkPlan ? SH::bytes - SH::off_prow : SH::bytes;
  auto kern = conv_packed_kernel<KS, NCT, MODE>;
  static std::once_flag once;
  static hipError_t err = hipSuccess;
  std::call_once(once, [&] {
    err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  });
  if (err != hipSuccess) return err;
  hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(SH::NT), (size_t)lds, stream, a);
  return hipGetLastError();
}

bool packed_channels_ok(int32_t C) { return C == 64 || C == 128; }

}  // namespace

bool conv_packed_supported(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout) {
  if (K < 1 || K > kPkMaxK) return false;
  if (!packed_channels_ok(Cin) || !packed_channels_ok(Cout)) return false;
  // chunks are counted in 32 bits
  return n_rows <= 0x7FFFFFFFLL;
}

int64_t conv_packed_weights_bytes(int32_t K, int32_t Cin, int32_t Cout) {
  return (int64_t)K * Cin * Cout * 2;
}

hipError_t launch_pack_conv_weights(const void* W, int32_t K, int32_t Cin, int32_t Cout,
                                    void* Wp, hipStream_t stream) {
  const int64_t total = (int64_t)K * (Cout / 16) * (Cin / 32) * 64;
  const unsigned blocks = (unsigned)((total + 255) / 256);
  hipLaunchKernelGGL(pack_weights_kernel, dim3(blocks), dim3(256), 0, stream,
                     static_cast<const uint16_t*>(W), K, Cin, Cout, static_cast<uint16_t*>(Wp));
  return hipGetLastError();
}

#define SHC_PACKED_SHAPES(X) X(64, 64) X(64, 128) X(128, 64) X(128, 128)

hipError_t launch_conv_packed(const void* S, const int32_t* table, int64_t n_rows, int32_t K,
                              const void* Wp, const float* bias, int32_t Cin, int32_t Cout,
                              int32_t relu, void* out, int num_cus, hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  PackedArgs a{};
  a.S = S;
  a.table = table;
  a.Wp = Wp;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.K = K;
  a.relu = relu;
#define SHC_PACKED_CASE(CI, CO)                                                              \
  if (Cin == CI && Cout == CO) return launch_packed_k<CI / 32, CO / 16, kPkFull>(a, num_cus, stream);
  SHC_PACKED_SHAPES(SHC_PACKED_CASE)
#undef SHC_PACKED_CASE
  return hipErrorInvalidValue;
}

int64_t conv_packed_plan_bytes(int64_t n_rows, int32_t Cin, int32_t Cout, int num_cus) {
  int32_t rc = 0, chunks = 0;
#define SHC_PACKED_CASE(CI, CO)                                                   \
  if (Cin == CI && Cout == CO) {                                                  \
    packed_chunks<CI / 32, CO / 16>(n_rows, num_cus, &rc, &chunks);               \
    return (int64_t)chunks * PkShape<CI / 32, CO / 16>::IMG;                      \
  }
  SHC_PACKED_SHAPES(SHC_PACKED_CASE)
#undef SHC_PACKED_CASE
  return 0;
}

int64_t conv_packed_plan_bytes_upto(int64_t n_rows, int32_t Cin, int32_t Cout, int num_cus) {
  // chunks(n) is at most max(CUs, ceil(n / RMAX)) for every n <= n_rows
  int64_t rmax = 0, img = 0;
#define SHC_PACKED_CASE(CI, CO)                                                   \
  if (Cin == CI && Cout == CO) {                                                  \
    rmax = PkShape<CI / 32, CO / 16>::RMAX;                                       \
    img = PkShape<CI / 32, CO / 16>::IMG;                                         \
  }
  SHC_PACKED_SHAPES(SHC_PACKED_CASE)
#undef SHC_PACKED_CASE
  if (img == 0) return 0;
  int64_t chunks = (n_rows + rmax - 1) / rmax;
  if (chunks < num_cus) chunks = num_cus;
  return chunks * img;
}

hipError_t launch_build_packed_plan(const int32_t* table, int64_t n_rows, int32_t K, int32_t Cin,
                                    int32_t Cout, void* plan, int num_cus, hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  PackedArgs a{};
  a.table = table;
  a.n_rows = n_rows;
  a.K = K;
  a.plan = plan;
#define SHC_PACKED_CASE(CI, CO)                                                              \
  if (Cin == CI && Cout == CO) return launch_packed_k<CI / 32, CO / 16, kPkPlan>(a, num_cus, stream);
  SHC_PACKED_SHAPES(SHC_PACKED_CASE)
#undef SHC_PACKED_CASE
  return hipErrorInvalidValue;
}

hipError_t launch_conv_packed_planned(const void* S, const void* plan, int64_t n_rows, int32_t K,
                                      const void* Wp, const float* bias, int32_t Cin,
                                      int32_t Cout, int32_t relu, void* out, int num_cus,
                                      hipStream_t stream) {
  if (n_rows == 0) return hipSuccess;
  PackedArgs a{};
  a.S = S;
  a.Wp = Wp;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.K = K;
  a.relu = relu;
  a.plan = const_cast<void*>(plan);
#define SHC_PACKED_CASE(CI, CO)                                                              \
  if (Cin == CI && Cout == CO)                                                               \
    return launch_packed_k<CI / 32, CO / 16, kPkPlanned>(a, num_cus, stream);
  SHC_PACKED_SHAPES(SHC_PACKED_CASE)
#undef SHC_PACKED_CASE
  return hipErrorInvalidValue;
}
#undef SHC_PACKED_SHAPES

}  // namespace shc
