// Sparse neighbourhood convolution from a neighbour-row table (Eqs. 4-5,
// with the activation of Eq. 10), bf16, slot-major:
//
//   out[i] = act( bias + sum_{j<K} S[table[j][i]] W[j] ),  absent entries add 0.
//
// A workgroup owns 128 or 256 consecutive active rows and every output
// column.  It walks the slots in order: the weights of slot j (Cin x Cout)
// sit in LDS while every wavefront multiplies its rows' slot-j neighbour rows
// by them, and slot j + 1's weights are loaded beside that work into the
// other of two buffers; the neighbour rows of slot j + 2 (and j + 1) are in
// flight in registers meanwhile.  Each gathered row therefore feeds all Cout
// columns at once, and the index work per row group is one pass over its
// table entries (no sort, no job lists).  A (16-row block, slot) pair with
// no present row is skipped.  Accumulation is in fp32, per output element
// in slot order and within a slot in k order.
#include <hip/hip_runtime.h>

#include <mutex>

#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kSmMaxSlots = 32;
constexpr int kSmLdsLimit = 160 * 1024;
constexpr int kSmBufferWord3 = 0x00020000;  // raw buffer resource, 32-bit data
constexpr uint32_t kSmOutOfRange = 0x80000000u;
#define SHC_SM_LDS __attribute__((address_space(3)))

typedef __bf16 sm_bf16x4 __attribute__((__vector_size__(4 * sizeof(__bf16))));
typedef __bf16 sm_bf16x2 __attribute__((ext_vector_type(2)));
typedef float sm_f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t sm_v4u32 __attribute__((ext_vector_type(4)));

// LDS: two weight buffers [Cin][Cout] bf16 (32-byte column chunks XOR-
// swizzled by row), srcs [K][R] int32, presence bytes [K][R/16], and one
// epilogue staging tile [16][Cout + 8] bf16 per wavefront.
__host__ __device__ constexpr int sm_wbuf_bytes(int cin, int cout) { return cin * cout * 2; }
__host__ __device__ constexpr int sm_stage_row(int cout) { return cout * 2 + 16; }
// srcs [K][R] in row order, then sorted; perm [R]; per-slot counts and the
// sort's buckets [K + 2]; presence bytes [K][R / 16]
__host__ __device__ inline int sm_idx_bytes(int K, int R) {
  return 4 * (2 * K * R + R + K + K + 2) + ((K * (R / 16) + 15) & ~15) + 16;
}
__host__ __device__ inline int sm_lds_bytes(int cin, int cout, int K, int R, int nw) {
  return 2 * sm_wbuf_bytes(cin, cout) + ((sm_idx_bytes(K, R) + 15) & ~15) +
         nw * 16 * sm_stage_row(cout);
}

struct SmArgs {
  const void* S;          // [n_rows][Cin] bf16
  const int32_t* table;   // [K][n_rows]
  const void* W;          // [K][Cin][Cout] bf16
  const float* bias;      // [Cout] or null
  void* out;              // [n_rows][Cout] bf16
  int64_t n_rows;
  int32_t K;
  int32_t relu;
};

// KS: 32-wide k-steps (Cin / 32); NCT: 16-column tiles (Cout / 16); NW:
// wavefronts per workgroup; BPW: 16-row blocks per wavefront (R = 16 NW BPW
// rows per workgroup); PD: slots of neighbour rows in flight ahead of the
// one being multiplied; KF: K fixed at compile time (the slots fully
// unrolled), or 0 for any K (a loop over the slots, whose back edge makes the
// compiler wait for every load in flight); WSET: register sets of weights
// (2: a slot's weights are loaded three slots ahead, 1: two).
template <int KS, int NCT, int NW, int BPW, int PD, int KF, int WSET>
__global__ __launch_bounds__(64 * NW, 1) void conv_sm_kernel(const SmArgs a) {
  constexpr int NT = 64 * NW;
  constexpr int Cin = KS * 32;
  constexpr int Cout = NCT * 16;
  constexpr int R = BPW * 16 * NW;
  constexpr int WROW = Cout * 2;           // weight row bytes in LDS
  constexpr int VPR = WROW / 16;           // 16-byte vectors per weight row
  constexpr int WVEC = Cin * VPR;          // vectors per slot's weights
  constexpr int NWV = WVEC / NT;           // per thread
  static_assert(WVEC % NT == 0, "whole weight vectors per thread");
  static_assert(R % 64 == 0, "a wavefront's 64 consecutive rows share a slot");
  constexpr int SROW = sm_stage_row(Cout);
  constexpr int NSET = PD + 1;             // register sets of neighbour rows

  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int K = KF > 0 ? KF : a.K;
  unsigned char* wbuf = smem;                                             // [2][Cin][WROW]
  int32_t* srcs_in = reinterpret_cast<int32_t*>(smem + 2 * sm_wbuf_bytes(Cin, Cout));  // [K][R]
  int32_t* srcs = srcs_in + K * R;        // [K][R], sorted positions
  int32_t* perm = srcs + K * R;           // [R] sorted position -> row
  int32_t* cnt = perm + R;                // [K] rows present per slot
  int32_t* hist = cnt + K;                // [K + 2] bucket counts, then cursors
  uint8_t* pres = reinterpret_cast<uint8_t*>(hist + K + 2);  // [K][R/16]
  unsigned char* stage = smem + 2 * sm_wbuf_bytes(Cin, Cout) + ((sm_idx_bytes(K, R) + 15) & ~15);

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int g = lane >> 4;
  const int l16 = lane & 15;
  const int64_t n = a.n_rows;
  const int64_t row0 = (int64_t)blockIdx.x * R;
  const int nrows = (int)min((int64_t)R, n - row0);

  // ---- weights of a slot: global -> registers -> LDS.  The 32-byte column
  // chunk c of weight row r sits at chunk position c ^ swz_row(r): a
  // transposing B read touches rows 8g + i (+4), g < 4, i < 4, and with
  // 256-byte rows (64 banks: every row starts on bank 0) the XOR puts the
  // eight rows of g & 1 and i at eight different banks groups; with 128-byte
  // rows (two rows per bank cycle) two bits of the row do it.
  auto swz_row = [](int r) -> int {
    if constexpr (NCT >= 8) return (r & 3) | (((r >> 3) & 1) << 2);
    else return ((r >> 1) & 1) | (((r >> 3) & 1) << 1);
  };
  const unsigned char* W = static_cast<const unsigned char*>(a.W);
  // slot m's weights are loaded WSET + 1 slots ahead of use (register set
  // m % WSET) and stored one slot ahead (buffer m & 1)
  static_assert(WSET == 1 || WSET == 2, "one or two register sets of weights");
  i32x4 wreg[WSET][NWV];
  auto load_w = [&](int j, i32x4 (&wr)[NWV]) {
#pragma unroll
    for (int u = 0; u < NWV; ++u) {
      const int v = u * NT + tid;
      wr[u] = *reinterpret_cast<const i32x4*>(W + ((int64_t)j * Cin * Cout) * 2 + v * 16);
    }
  };
  auto store_w = [&](int buf, const i32x4 (&wr)[NWV]) {
    unsigned char* base = wbuf + buf * sm_wbuf_bytes(Cin, Cout);
#pragma unroll
    for (int u = 0; u < NWV; ++u) {
      const int v = u * NT + tid;
      const int k = v / VPR;
      const int q = v - k * VPR;
      const int col = (((q >> 1) ^ swz_row(k)) << 5) + ((q & 1) << 4);
      *reinterpret_cast<i32x4*>(base + k * WROW + col) = wr[u];
    }
  };
  // B fragments of one k-step (rows 32 ks .. 32 ks + 31) from a buffer: two
  // transposing reads per 16 columns give lane (g, i) rows 8g .. 8g+7 of
  // column i; the lane's rows 32 ks + 8g + (i >> 2) and 4 more share one
  // swizzle, a per-lane constant
  const int swz = swz_row(8 * g + (l16 >> 2));
  auto read_b = [&](int buf, int ks, bf16x8* out) {
    const unsigned char* base = wbuf + buf * sm_wbuf_bytes(Cin, Cout) + ks * 32 * WROW;
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
      const unsigned char* p0 =
          base + (8 * g + (l16 >> 2)) * WROW + (((ct ^ swz) << 5) + 8 * (l16 & 3));
      const sm_bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (SHC_SM_LDS sm_bf16x4*)(const_cast<unsigned char*>(p0)));
      const sm_bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
          (SHC_SM_LDS sm_bf16x4*)(const_cast<unsigned char*>(p0 + 4 * WROW)));
      out[ct] = bf16x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
  };

  // ---- prologue: slot 0's weights on their way, then the table entries
  load_w(0, wreg[0]);
  for (int q = tid; q < 2 * K + 2; q += NT) cnt[q] = 0;  // cnt and hist
  __syncthreads();
  // entries (j, t) = (e / R, e % R): a wavefront reads 64 consecutive rows of
  // one slot, coalesced, eight entries per thread in flight
  const int KR = K * R;
  for (int e0 = 0; e0 < KR; e0 += 8 * NT) {
    int32_t s[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + u * NT + tid;
      const int j = e / R, t = e - (e / R) * R;
      s[u] = (e < KR && t < nrows) ? a.table[(int64_t)j * n + row0 + t] : -1;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + u * NT + tid;
      const bool ok = (uint32_t)s[u] < (uint32_t)n;  // 0 <= s < n
      const int c = __popcll(__ballot(ok));
      if (e < KR) {
        srcs_in[e] = ok ? s[u] : -1;
        if (lane == 0 && c > 0) atomicAdd(&cnt[e / R], c);
      }
    }
  }
  __syncthreads();
  // Rows sorted by their first sparse slot (a slot present in fewer than
  // half the rows), so that rows sharing it share 16-row blocks and a
  // block's slot is more often present in none of its rows: a counting sort
  // over buckets 0 (dense slots only), 1 + j (first sparse slot j), K + 1
  // (past the last row); the order inside a bucket is whatever the atomics
  // give, which no result depends on (every row's sum runs over its own
  // slots in order).
  constexpr int RPT = (R + NT - 1) / NT;  // rows per thread
  int bkt[RPT];
  uint32_t dense = 0;
  for (int j = 0; j < K; ++j) dense |= (2 * cnt[j] >= nrows ? 1u : 0u) << j;
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int t = tid + i * NT;
    bkt[i] = -1;
    if (t < R) {
      uint32_t rm = 0;
      for (int j = 0; j < K; ++j) rm |= (srcs_in[j * R + t] >= 0 ? 1u : 0u) << j;
      const uint32_t key = rm & ~dense;
      bkt[i] = t >= nrows ? K + 1 : (key ? 1 + __builtin_ctz(key) : 0);
      atomicAdd(&hist[bkt[i]], 1);
    }
  }
  __syncthreads();
  if (wave == 0) {  // exclusive scan of the K + 2 <= 34 counts, one per lane
    const int c = lane < K + 2 ? hist[lane] : 0;
    int inc = c;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const int y = __shfl_up(inc, d, 64);
      if (lane >= d) inc += y;
    }
    if (lane < K + 2) hist[lane] = inc - c;
  }
  __syncthreads();
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int t = tid + i * NT;
    if (t < R) {
      const int pos = atomicAdd(&hist[bkt[i]], 1);
      perm[pos] = t;
      for (int j = 0; j < K; ++j) srcs[j * R + pos] = srcs_in[j * R + t];
    }
  }
  __syncthreads();
  // presence of each (slot, sorted 16-row block)
  for (int e = tid; e < KR; e += NT) {
    const uint64_t bal = __ballot(srcs[e] >= 0);
    if (l16 == 0) pres[(e / R) * (R / 16) + (e % R) / 16] = ((bal >> (lane & 48)) & 0xFFFFu) != 0;
  }
  store_w(0, wreg[0]);
  __syncthreads();

  // ---- neighbour rows of a slot for this wavefront's blocks: raw buffer
  // loads, an absent row reading zeros without touching memory
  const __amdgpu_buffer_rsrc_t s_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(a.S), (short)0, (int)(n * Cin * 2), kSmBufferWord3);
  i32x4 areg[NSET][BPW][KS];
  auto issue_a = [&](int j, i32x4 (&dst)[BPW][KS]) {
#pragma unroll
    for (int u = 0; u < BPW; ++u) {
      const int row = (wave * BPW + u) * 16 + l16;
      const int32_t src = j < K ? srcs[j * R + row] : -1;
      const uint32_t off = src >= 0 ? (uint32_t)src * (uint32_t)(Cin * 2) + (uint32_t)g * 16u
                                    : kSmOutOfRange;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks)
        dst[u][ks] = __builtin_bit_cast(
            i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                       s_rsrc, src >= 0 ? off + (uint32_t)ks * 64u : kSmOutOfRange, 0, 0));
    }
  };

  // accumulators start at the bias of their column
  f32x4 acc[BPW][NCT];
#pragma unroll
  for (int ct = 0; ct < NCT; ++ct) {
    const float b = a.bias != nullptr ? a.bias[ct * 16 + l16] : 0.f;
#pragma unroll
    for (int u = 0; u < BPW; ++u) acc[u][ct] = f32x4{b, b, b, b};
  }

  // loads go out in the loop's own order (weights of slot m + 3 beside the
  // rows of slot m + PD), so that every slot's waits count the same loads
  static_assert(PD == 1 || PD == 2, "one or two slots of rows ahead");
  issue_a(0, areg[0]);
  load_w(K > 1 ? 1 : K - 1, wreg[1 % WSET]);
  if constexpr (PD == 2) issue_a(1, areg[1]);
  if constexpr (WSET == 2) load_w(K > 2 ? 2 : K - 1, wreg[0]);

  // ---- the slots, in order; register set j % NSET, weight buffer j % 2
  auto slot = [&](int j, i32x4 (&cur)[BPW][KS], i32x4 (&ahead)[BPW][KS], i32x4 (&wr)[NWV]) {
    // slot j's weights were stored before this barrier; every wavefront is
    // done with slot j - 1, so its buffer takes slot j + 1's (register set
    // (j + 1) & 1, which then loads slot j + 3's).  Past the last slot the
    // weights of slot K - 1 are loaded and stored again, into a buffer no
    // slot reads any more, so that every slot issues the same loads.
    __syncthreads();
    store_w((j + 1) & 1, wr);
    load_w(j + WSET + 1 < K ? j + WSET + 1 : K - 1, wr);
    issue_a(j + PD, ahead);
    bool live[BPW];
    bool any = false;
#pragma unroll
    for (int u = 0; u < BPW; ++u) {
      live[u] = pres[j * (R / 16) + wave * BPW + u] != 0;
      any = any || live[u];
    }
    if (!any) return;  // no row of this wavefront has slot j: no B reads either
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      bf16x8 bfr[NCT];
      read_b(j & 1, ks, bfr);
#pragma unroll
      for (int u = 0; u < BPW; ++u) {
        if (!live[u]) continue;
        const bf16x8 af = __builtin_bit_cast(bf16x8, cur[u][ks]);
#pragma unroll
        for (int ct = 0; ct < NCT; ++ct)
          acc[u][ct] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af, bfr[ct], acc[u][ct], 0, 0, 0);
      }
    }
  };
  if constexpr (KF > 0) {
#pragma unroll
    for (int j = 0; j < KF; ++j)
      slot(j, areg[j % NSET], areg[(j + PD) % NSET], wreg[(j + 1) % WSET]);
  } else {
    // six slots per trip: register sets j % NSET and weight sets (j + 1) % 2
    for (int j0 = 0; j0 < K; j0 += 6) {
#pragma unroll
      for (int p = 0; p < 6; ++p)
        if (j0 + p < K)
          slot(j0 + p, areg[p % NSET], areg[(p + PD) % NSET], wreg[(p + 1) % WSET]);
    }
  }

  // ---- epilogue: act, bf16 (round to nearest even), staged per wavefront
  // so that every lane stores 16 contiguous bytes of a row
  __builtin_amdgcn_sched_barrier(0);
  const bool relu = a.relu != 0;
  unsigned char* my_stage = stage + wave * 16 * SROW;
  const __amdgpu_buffer_rsrc_t o_rsrc = __builtin_amdgcn_make_buffer_rsrc(
      a.out, (short)0, (int)(n * Cout * 2), kSmBufferWord3);
#pragma unroll
  for (int u = 0; u < BPW; ++u) {
#pragma unroll
    for (int ct = 0; ct < NCT; ++ct) {
      float v[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float x = acc[u][ct][r];
        const float rx = x > 0.f ? x : 0.f;
        v[r] = relu ? rx : x;
      }
      unsigned char* pp = my_stage + (g * 4) * SROW + (ct * 16 + l16) * 2;
#pragma unroll
      for (int r = 0; r < 4; r += 2) {
        const sm_bf16x2 h = __builtin_convertvector(sm_f32x2{v[r], v[r + 1]}, sm_bf16x2);
        *reinterpret_cast<__bf16*>(pp + r * SROW) = h[0];
        *reinterpret_cast<__bf16*>(pp + (r + 1) * SROW) = h[1];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    constexpr int NST = 16 * VPR / 64;  // 16-byte stores per lane for the block
    i32x4 sv[NST];
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int idx = t * 64 + lane;
      sv[t] = *reinterpret_cast<const i32x4*>(my_stage + (idx / VPR) * SROW + (idx % VPR) * 16);
    }
    int prow[NST];
#pragma unroll
    for (int t = 0; t < NST; ++t) prow[t] = perm[(wave * BPW + u) * 16 + (t * 64 + lane) / VPR];
#pragma unroll
    for (int t = 0; t < NST; ++t) {
      const int idx = t * 64 + lane;
      const int r = prow[t];
      const uint32_t off = r < nrows
                               ? ((uint32_t)(row0 + r) * (uint32_t)Cout + (uint32_t)(idx % VPR) * 8u) * 2u
                               : kSmOutOfRange;
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(sm_v4u32, sv[t]), o_rsrc, off, 0,
                                             0);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

template <int KS, int NCT, int NW, int BPW, int PD, int KF>
hipError_t launch_sm(const SmArgs& a, hipStream_t stream) {
  constexpr int R = BPW * 16 * NW;
  // one wavefront per SIMD keeps five blocks' accumulators and rows in
  // registers, with one register set of weights
  auto kern = conv_sm_kernel<KS, NCT, NW, BPW, PD, KF, NW >= 8 ? 2 : 1>;
  static std::once_flag once;
  static hipError_t attr_err = hipSuccess;
  std::call_once(once, [&] {
    attr_err = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                   hipFuncAttributeMaxDynamicSharedMemorySize, kSmLdsLimit);
  });
  if (attr_err != hipSuccess) return attr_err;
  const size_t lds = (size_t)sm_lds_bytes(KS * 32, NCT * 16, a.K, R, NW);
  const unsigned grid = (unsigned)((a.n_rows + R - 1) / R);
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * NW), lds, stream, a);
  return hipGetLastError();
}

// Rows per workgroup (one workgroup per CU: the LDS holds one): the fewest
// of 128 (8 wavefronts x 1 block), 256 (8 x 2) and 320 (4 x 5, one
// wavefront per SIMD holding all five blocks' accumulators and rows) that
// covers the rows in one round, else 256 (nine slots) or 320.  The 8-wavefront
// kernels run nine slots unrolled and two slots of rows ahead; the others
// loop over the slots (whose back edge waits for every load, which with one
// slot of rows ahead is about what the next slot waits for anyway).
template <int KS, int NCT>
hipError_t launch_sm_rows(const SmArgs& a, int num_cus, hipStream_t stream) {
  const int64_t n = a.n_rows;
  const bool k9 = a.K == 9;
  if ((n + 127) / 128 <= num_cus)
    return k9 ? launch_sm<KS, NCT, 8, 1, 2, 9>(a, stream) : launch_sm<KS, NCT, 8, 1, 2, 0>(a, stream);
  if (k9 && (n + 255) / 256 <= num_cus) return launch_sm<KS, NCT, 8, 2, 2, 9>(a, stream);
  if ((n + 319) / 320 <= num_cus || !k9) return launch_sm<KS, NCT, 4, 5, 1, 0>(a, stream);
  return launch_sm<KS, NCT, 8, 2, 2, 9>(a, stream);
}

}  // namespace

bool conv_sm_supported(const GemmArgs& a, bool bf16) {
  if (!bf16 || a.table == nullptr || a.plan != nullptr || a.plan_out != nullptr || a.gather)
    return false;
  if (a.K < 1 || a.K > kSmMaxSlots) return false;
  if (!((a.Cin == 64 || a.Cin == 128) && (a.Cout == 64 || a.Cout == 128))) return false;
  // 32-bit buffer offsets
  if (a.n_rows * a.Cin * 2 > 0x7FFF0000LL || a.n_rows * a.Cout * 2 > 0x7FFF0000LL) return false;
  return sm_lds_bytes(a.Cin, a.Cout, a.K, 320, 4) <= kSmLdsLimit &&
         sm_lds_bytes(a.Cin, a.Cout, a.K, 256, 8) <= kSmLdsLimit;
}

hipError_t launch_conv_sm(const GemmArgs& g, int num_cus, hipStream_t stream) {
  SmArgs a;
  a.S = g.S;
  a.table = g.table;
  a.W = g.W;
  a.bias = g.bias;
  a.out = g.out;
  a.n_rows = g.n_rows;
  a.K = g.K;
  a.relu = g.relu;
  if (a.n_rows == 0) return hipSuccess;
  if (g.Cin == 128 && g.Cout == 128) return launch_sm_rows<4, 8>(a, num_cus, stream);
  if (g.Cin == 128 && g.Cout == 64) return launch_sm_rows<4, 4>(a, num_cus, stream);
  if (g.Cin == 64 && g.Cout == 128) return launch_sm_rows<2, 8>(a, num_cus, stream);
  if (g.Cin == 64 && g.Cout == 64) return launch_sm_rows<2, 4>(a, num_cus, stream);
  return hipErrorInvalidValue;
}

}  // namespace shc
