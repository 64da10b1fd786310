// Internal declarations shared by the HIP translation units of libshc.so.
// Nothing here is part of the public ABI (include/shc.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace shc {

// ---------------------------------------------------------------------------
// small device helpers
// ---------------------------------------------------------------------------

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ float bf16_bits_to_f32(uint32_t h) {
  return __uint_as_float(h << 16);
}

// fp32 -> bf16 bits, round to nearest, ties to even; NaN -> quiet NaN.
// Adding 0x7FFF plus the lowest kept bit to the fp32 pattern carries into the
// kept part exactly when the dropped half is above one half ulp, or equal to
// it with an odd kept part.
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0u | ((u >> 16) & 0x8000u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

template <typename T>
__device__ __forceinline__ T ceil_div(T a, T b) {
  return (a + b - 1) / b;
}

// ---------------------------------------------------------------------------
// launchers (host side, enqueue only; arguments already validated)
// ---------------------------------------------------------------------------

// the calling thread's last-error message (shc_last_error), for entry points
// defined outside the file that owns it; set_error returns `code`
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

// compaction: number of blocks and per-block element span for a mask of `total` entries
void compact_plan(int64_t total, int32_t* nblocks, int64_t* per_block);

hipError_t launch_compact(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords, int32_t* inv,
                          int32_t* row_ptr, int32_t* n_active, int64_t* n_host, int64_t cap,
                          int32_t* block_counts, hipStream_t stream);

// compaction that also writes the neighbour-row table of the active set
// (table[j * N' + i], as launch_neighbor_table), one block per body: the body's
// row numbering lives in LDS, 8 bytes per vertex
constexpr int32_t kCompactTableMaxV = 19456;
bool compact_table_supported(int32_t V, int32_t K);
hipError_t launch_compact_table(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                                int32_t* inv, int32_t* row_ptr, int32_t* n_active,
                                int64_t* n_host, int64_t cap, const int32_t* nbr, int32_t K,
                                int32_t* table, int32_t* block_counts, hipStream_t stream);

hipError_t launch_gather(const void* x, const int32_t* coords, int64_t n_rows, int32_t B,
                         int32_t V, int32_t row_bytes, void* S, hipStream_t stream);

int group_norm_split(int32_t B, int32_t C, int32_t G, int is_bf16, int num_cus);
size_t group_norm_lds_bytes(int32_t C, int is_bf16, int split);
hipError_t launch_group_norm(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                             int32_t C, int32_t G, float eps, int is_bf16, void* out,
                             int num_cus, hipStream_t stream);
// mask scores (scores.hip)
constexpr int kMaxScoreMasks = 64;
void mask_scores_plan(int32_t K, int64_t N, int32_t C, int* tile, int* tiles, int* splits,
                      int64_t* rows_per_split, int* chunks);
size_t mask_scores_workspace_bytes(int32_t K, int64_t N, int32_t C);
hipError_t launch_mask_scores(const void* O, int32_t K, int64_t N, int32_t C,
                              const double* alpha_in, double* alpha_out, double* sim,
                              int32_t kappa, int32_t* top, void* ws, hipStream_t stream);
// backward of the linear and conv layers (backward.hip)
constexpr int kMaxVirtualSlots = 64;
struct BwdPlan {
  int T, tiles, L, splits;
  int64_t max_chunks, rps;
  size_t off_dz, off_colpart, off_pairs, off_rowptr, off_mask, off_part, total;
};
void backward_plan(int64_t n, int32_t K, int32_t Cin, int32_t Cout, int is_bf16, int conv,
                   BwdPlan* p);
int backward_dgrad_supported(int32_t Kw, int32_t Cin, int32_t Cout, int is_bf16);
size_t transpose_neighbors_ws_bytes(int32_t V, int32_t K);
hipError_t launch_transpose_neighbors(const int32_t* nbr, int32_t V, int32_t K, int32_t* nbr_t,
                                      int32_t* slot_of, int32_t* off_dev, void* ws,
                                      hipStream_t stream);
hipError_t launch_transposed_table(const int32_t* coords, const int32_t* inv, int64_t n, int32_t B,
                                   int32_t V, const int32_t* nbr_t, int32_t Kt, int32_t* table_t,
                                   uint64_t* row_slots, hipStream_t stream);
hipError_t launch_fill_i32(int32_t* p, int64_t n, int32_t v, hipStream_t stream);
size_t slot_pairs_ws_bytes(int64_t n, int32_t K);
hipError_t launch_slot_pairs(const int32_t* table, int64_t n, int32_t K, int32_t* pairs,
                             int32_t* pair_ptr, void* ws, hipStream_t stream);
hipError_t launch_layer_backward(int conv, const void* S, const int32_t* table,
                                 const int32_t* pairs, const int32_t* pair_ptr,
                                 const int32_t* table_t, const uint64_t* row_slots,
                                 const int32_t* slot_of, const void* W, const void* Y,
                                 const void* dY, int64_t n, int32_t K, int32_t Cin, int32_t Cout,
                                 int is_bf16, int act, void* dS, float* dW, float* db, void* ws,
                                 hipStream_t stream);
hipError_t launch_clear_inactive(const int32_t* inv, int32_t B, int32_t V, int32_t row_bytes,
                                 void* D, hipStream_t stream);
hipError_t launch_scatter_update(const void* S, const int32_t* inv, const int32_t* coords,
                                 int64_t n_rows, const int32_t* prev_coords, int64_t prev_rows,
                                 int32_t B, int32_t V, int32_t row_bytes, void* D,
                                 hipStream_t stream);
hipError_t launch_gather_ext(const void* x, const uint8_t* me, int mask_mode,
                             const int32_t* coords, int64_t n_rows, int32_t B, int32_t Bx,
                             int32_t V, int32_t row_bytes, void* S, hipStream_t stream);
hipError_t launch_combine(const void* Y, int32_t kappa, int64_t rows, int32_t row_bytes, int op,
                          int is_bf16, void* out, hipStream_t stream);
hipError_t launch_row_activity(const uint8_t* me, int32_t B, int32_t V, int32_t C, uint8_t* m,
                               hipStream_t stream);
hipError_t launch_scatter(const void* S, const int32_t* inv, const int32_t* coords,
                          int64_t n_rows, int32_t B, int32_t V, int32_t row_bytes, int zero_fill,
                          void* D, hipStream_t stream);

hipError_t launch_segment_max(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                              int32_t C, int is_bf16, float empty_value, void* P,
                              hipStream_t stream);

// neighbour-row table of the active set: table[j * n_rows + i] = row of slot j's
// neighbour of active row i, or -1
hipError_t launch_neighbor_table(const int32_t* coords, const int32_t* inv, int64_t n_rows,
                                 int32_t B, int32_t V, const int32_t* nbr, int32_t K,
                                 int32_t* table, hipStream_t stream);

struct GemmArgs {
  const void* S;        // [n_rows][Cin]
  const int32_t* coords;  // conv only
  const int32_t* inv;     // conv only
  const int32_t* nbr;     // conv only, [V][K]
  const int32_t* table;   // conv from a neighbour-row table, [K][n_rows]; else null
  const void* W;        // [K][Cin][Cout] (linear: K = 1)
  const float* bias;    // [Cout] or null
  void* out;            // [n_rows][Cout]
  int64_t n_rows;
  int32_t B, V, K, Cin, Cout;
  int32_t relu;
  int32_t gather;       // linear only: input row i is S[coords b_i * V + v_i] (S = dense x)
  uint32_t cin_magic;   // ceil(2^32 / Cin), filled in by the launcher
  // conv from a table, weight-stationary kernel only: write the active set's
  // plan (index lists, sort, job lists per row group) to plan_out instead of
  // computing, or read it from plan; images plan_stride bytes apart
  void* plan_out;
  const void* plan;
  int64_t plan_stride;
};

hipError_t launch_gather_gemm(const GemmArgs& a, bool conv, bool bf16, hipStream_t stream);

// weight-stationary variant (conv_ws.hip): LDS plan, all sizes in bytes
struct WsPlan {
  int ws;         // output-column slice width held in LDS
  int wrow;       // padded LDS row of the weight slice
  int wbytes;     // weight slice
  int rows;       // active rows per workgroup (multiple of 16)
  int idx_bytes;  // index lists
  int scratch;    // epilogue staging (all waves)
  int total;
};
bool ws_plan(const GemmArgs& a, bool conv, bool bf16, int num_cus, WsPlan* plan);
// Bytes of the plan of a conv from a table with this shape (0: the shape
// takes no plan), and the distance between two row groups' images.
int64_t conv_plan_bytes(const GemmArgs& a, bool bf16, int num_cus, int64_t* stride);
// The largest row count whose conv takes a plan (0: none), and the largest
// plan of any row count up to a.n_rows.
int64_t conv_plan_max_rows(const GemmArgs& a, bool bf16, int num_cus);
int64_t conv_plan_bytes_upto(const GemmArgs& a, bool bf16, int num_cus);
hipError_t launch_ws_gemm(const GemmArgs& a, bool conv, bool bf16, const WsPlan& plan,
                          hipStream_t stream);
// slot-major conv from a neighbour-row table (conv_sm.hip): bf16, C_in and
// C_out in {64, 128}, K <= 32, no plan
bool conv_sm_supported(const GemmArgs& a, bool bf16);
hipError_t launch_conv_sm(const GemmArgs& a, int num_cus, hipStream_t stream);
// conv from a neighbour-row table with slot 0 and the other slots apart
// (conv_split.hip): bf16, C_in and C_out in {64, 128, 256}, K <= 32; the
// other slots' partial rows go through an fp32 workspace of
// conv_split_workspace_bytes bytes
int64_t conv_split_workspace_bytes(int64_t n_rows, int32_t K, int32_t Cout);
bool conv_split_supported(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout);
hipError_t launch_conv_split(const void* S, const int32_t* table, int64_t n_rows, int32_t K,
                             const void* W, const float* bias, int32_t Cin, int32_t Cout,
                             int32_t relu, void* out, float* workspace, int num_cus,
                             hipStream_t stream);

// conv from a neighbour-row table with every slot's weights in registers
// (conv_packed.hip): bf16, C_in and C_out in {64, 128}, K <= 9, weights
// pre-arranged by launch_pack_conv_weights into conv_packed_weights_bytes
bool conv_packed_supported(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout);
int64_t conv_packed_weights_bytes(int32_t K, int32_t Cin, int32_t Cout);
hipError_t launch_pack_conv_weights(const void* W, int32_t K, int32_t Cin, int32_t Cout,
                                    void* Wp, hipStream_t stream);
hipError_t launch_conv_packed(const void* S, const int32_t* table, int64_t n_rows, int32_t K,
                              const void* Wp, const float* bias, int32_t Cin, int32_t Cout,
                              int32_t relu, void* out, int num_cus, hipStream_t stream);
// its plan: the rows' grouping and slot entries of every chunk, built once per
// active set (launch_build_packed_plan) and read by every packed layer of the
// shape (launch_conv_packed_planned)
int64_t conv_packed_plan_bytes(int64_t n_rows, int32_t Cin, int32_t Cout, int num_cus);
int64_t conv_packed_plan_bytes_upto(int64_t n_rows, int32_t Cin, int32_t Cout, int num_cus);
hipError_t launch_build_packed_plan(const int32_t* table, int64_t n_rows, int32_t K, int32_t Cin,
                                    int32_t Cout, void* plan, int num_cus, hipStream_t stream);
hipError_t launch_conv_packed_planned(const void* S, const void* plan, int64_t n_rows, int32_t K,
                                      const void* Wp, const float* bias, int32_t Cin,
                                      int32_t Cout, int32_t relu, void* out, int num_cus,
                                      hipStream_t stream);

}  // namespace shc
