// Neighbour-row table of an active set: for active row i = (b_i, v_i) and
// kernel slot j, the compact row that slot j reads in the sparse
// convolution of Eqs. 4-5,
//
//   table[j * n_rows + i] = inv[b_i * V + nbr[v_i * K + j]],
//
// or -1 when the slot has no neighbour (nbr = -1, or out of range) or the
// neighbour vertex is not active in body b_i.  The active set is the same for
// every layer (C'_k = C_k), so one table serves every convolution on it.
//
// Slot-major layout: a run of rows of one slot is contiguous, so a consumer
// reading rows [r0, r0 + R) of every slot issues K fully coalesced segments.
// One thread per active row: it loads its coordinate once, then all K
// neighbour vertices, then all K inverse-map entries (each round fully in
// flight; addresses clamped, results masked after), and stores slot j of
// consecutive rows from consecutive lanes.
#include "shc_internal.h"

namespace shc {
namespace {

constexpr int kThreads = 256;

// KM >= K slots held per thread
template <int KM>
__global__ __launch_bounds__(kThreads) void neighbor_table_kernel(
    const int2* __restrict__ coords, const int32_t* __restrict__ inv, int64_t n_rows, int32_t B,
    int32_t V, const int32_t* __restrict__ nbr, int32_t K, int32_t* __restrict__ table) {
  const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  if (i >= n_rows) return;
  const int2 c = coords[i];
  const bool ok = c.x >= 0 && c.x < B && c.y >= 0 && c.y < V;
  const int32_t* nrow = nbr + (int64_t)(ok ? c.y : 0) * K;
  const int32_t* irow = inv + (int64_t)(ok ? c.x : 0) * V;
  int32_t u[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) u[j] = nrow[j < K ? j : K - 1];
#pragma unroll
  for (int j = 0; j < KM; ++j) u[j] = (ok && u[j] >= 0 && u[j] < V) ? u[j] : -1;
  int32_t r[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) r[j] = irow[u[j] >= 0 ? u[j] : 0];
#pragma unroll
  for (int j = 0; j < KM; ++j)
    if (j < K) table[(int64_t)j * n_rows + i] = (u[j] >= 0 && r[j] >= 0 && (int64_t)r[j] < n_rows) ? r[j] : -1;
}

}  // namespace

hipError_t launch_neighbor_table(const int32_t* coords, const int32_t* inv, int64_t n_rows,
                                 int32_t B, int32_t V, const int32_t* nbr, int32_t K,
                                 int32_t* table, hipStream_t stream) {
  if (n_rows <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n_rows + kThreads - 1) / kThreads);
  const int2* c = reinterpret_cast<const int2*>(coords);
  if (K <= 10)
    hipLaunchKernelGGL(neighbor_table_kernel<10>, dim3(blocks), dim3(kThreads), 0, stream, c, inv,
                       n_rows, B, V, nbr, K, table);
  else
    hipLaunchKernelGGL(neighbor_table_kernel<32>, dim3(blocks), dim3(kThreads), 0, stream, c, inv,
                       n_rows, B, V, nbr, K, table);
  return hipGetLastError();
}

}  // namespace shc
