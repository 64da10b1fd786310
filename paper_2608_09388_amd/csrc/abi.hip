// C ABI of libshc.so: argument validation on the host, then kernel launches.
// Validation never touches the device, so every error path can be exercised
// without a GPU.
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "../../include/shc.h"
#include <cmath>
#include <mutex>

#include "shc_internal.h"

namespace {

thread_local char g_last_error[512] = "";

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}

int hip_status(hipError_t err, const char* where) {
  if (err == hipSuccess) return SHC_OK;
  return fail(SHC_ERR_HIP, "%s: %s (%d)", where, hipGetErrorString(err), (int)err);
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int32_t kMaxChannels = 4096;
constexpr int32_t kMaxSlots = 32;

int check_dtype(int32_t dtype) {
  if (dtype != SHC_F32 && dtype != SHC_BF16)
    return fail(SHC_ERR_UNSUPPORTED, "unknown dtype code %d", dtype);
  return SHC_OK;
}

int check_channels(const char* name, int32_t C) {
  if (C <= 0) return fail(SHC_ERR_INVALID_ARG, "%s = %d must be positive", name, C);
  if (C % 16 != 0 || C > kMaxChannels)
    return fail(SHC_ERR_UNSUPPORTED, "%s = %d must be a multiple of 16 in [16, %d]", name, C,
                kMaxChannels);
  return SHC_OK;
}

int check_bv(int32_t B, int32_t V) {
  if (B <= 0 || V <= 0) return fail(SHC_ERR_INVALID_ARG, "B = %d and V = %d must be positive", B, V);
  if ((int64_t)B * V > INT32_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "B * V = %lld exceeds 2^31 - 1", (long long)B * V);
  return SHC_OK;
}

int check_rows(int64_t n_rows) {
  if (n_rows < 0 || n_rows > INT32_MAX)
    return fail(SHC_ERR_INVALID_ARG, "n_rows = %lld outside [0, 2^31)", (long long)n_rows);
  return SHC_OK;
}

#define SHC_TRY(expr)          \
  do {                         \
    int _rc = (expr);          \
    if (_rc != SHC_OK) return _rc; \
  } while (0)

#define SHC_PTR(p, name)                                                           \
  do {                                                                             \
    if ((p) == nullptr) return fail(SHC_ERR_INVALID_ARG, "%s is NULL", name);      \
    if (!aligned16(p)) return fail(SHC_ERR_MISALIGNED, "%s is not 16-byte aligned", name); \
  } while (0)

#define SHC_OPT_PTR(p, name)                                                       \
  do {                                                                             \
    if ((p) != nullptr && !aligned16(p))                                           \
      return fail(SHC_ERR_MISALIGNED, "%s is not 16-byte aligned", name);          \
  } while (0)

}  // namespace

namespace shc {
// The thread's last-error message, for entry points defined in other files.
int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
  va_end(ap);
  return code;
}
void clear_error() { g_last_error[0] = 0; }
}  // namespace shc

extern "C" {

const char* shc_status_string(int status) {
  switch (status) {
    case SHC_OK: return "SHC_OK";
    case SHC_ERR_INVALID_ARG: return "SHC_ERR_INVALID_ARG";
    case SHC_ERR_CAPACITY: return "SHC_ERR_CAPACITY";
    case SHC_ERR_MISALIGNED: return "SHC_ERR_MISALIGNED";
    case SHC_ERR_UNSUPPORTED: return "SHC_ERR_UNSUPPORTED";
    case SHC_ERR_HIP: return "SHC_ERR_HIP";
    default: return "SHC_ERR_UNKNOWN";
  }
}

const char* shc_last_error(void) { return g_last_error; }

size_t shc_compact_mask_workspace(int32_t B, int32_t V) {
  if (B <= 0 || V <= 0) return 0;
  int32_t nblocks;
  int64_t per_block;
  shc::compact_plan((int64_t)B * V, &nblocks, &per_block);
  return (((size_t)nblocks * sizeof(int32_t)) + 255u) & ~(size_t)255u;
}

// Device address of a caller's host variable when it lies in page-locked
// memory mapped into the device's address space, else null (pageable memory).
static int64_t* mapped_host_count(int64_t* host) {
  hipPointerAttribute_t attr;
  if (hipPointerGetAttributes(&attr, host) != hipSuccess) {
    (void)hipGetLastError();  // pageable memory: clear the lookup's error
    return nullptr;
  }
  if (attr.type != hipMemoryTypeHost || attr.devicePointer == nullptr) return nullptr;
  return static_cast<int64_t*>(attr.devicePointer);
}

// Validation and launch shared by shc_compact_mask and shc_compact_mask_start.
// *mapped receives the device address of a page-locked host count, or null
// (no host count, or pageable memory: refused when require_mapped).
// With nbr != NULL the neighbour-row table is written too (compact + table).
static int compact_launch(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords, int32_t* inv,
                          int32_t* row_ptr, int32_t* n_active_dev, int64_t* n_active_host,
                          bool require_mapped, int64_t** mapped_out, int64_t cap, void* ws,
                          size_t ws_bytes, hipStream_t stream, const int32_t* nbr = nullptr,
                          int32_t K = 0, int32_t* table = nullptr) {
  *mapped_out = nullptr;
  if (require_mapped && n_active_host == nullptr)
    return fail(SHC_ERR_INVALID_ARG, "n_active_host is NULL");
  SHC_TRY(check_bv(B, V));
  SHC_PTR(mask, "mask");
  SHC_PTR(inv, "inv");
  SHC_PTR(row_ptr, "row_ptr");
  SHC_PTR(n_active_dev, "n_active_dev");
  SHC_PTR(ws, "ws");
  if (cap < 0) return fail(SHC_ERR_INVALID_ARG, "cap = %lld is negative", (long long)cap);
  if (cap > 0) SHC_PTR(coords, "coords");
  const size_t need = shc_compact_mask_workspace(B, V);
  if (ws_bytes < need)
    return fail(SHC_ERR_CAPACITY, "workspace of %zu bytes is below the %zu needed", ws_bytes, need);
  int64_t* mapped = n_active_host ? mapped_host_count(n_active_host) : nullptr;
  if (require_mapped && mapped == nullptr)
    return fail(SHC_ERR_INVALID_ARG, "n_active_host is not page-locked host memory mapped "
                                     "into the device");
  *mapped_out = mapped;
  if (mapped != nullptr) *reinterpret_cast<volatile int64_t*>(n_active_host) = -1;  // set by the kernel
  if (nbr != nullptr)
    return hip_status(shc::launch_compact_table(mask, B, V, coords, inv, row_ptr, n_active_dev,
                                                mapped, cap, nbr, K, table,
                                                static_cast<int32_t*>(ws), stream),
                      "compact_mask_table launch");
  return hip_status(shc::launch_compact(mask, B, V, coords, inv, row_ptr, n_active_dev, mapped,
                                        cap, static_cast<int32_t*>(ws), stream),
                    "compact_mask launch");
}

int shc_compact_mask_start(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                           int32_t* inv, int32_t* row_ptr, int32_t* n_active_dev,
                           int64_t* n_active_host, int64_t cap, void* ws, size_t ws_bytes,
                           hipStream_t stream) {
  g_last_error[0] = 0;
  int64_t* mapped = nullptr;
  return compact_launch(mask, B, V, coords, inv, row_ptr, n_active_dev, n_active_host, true,
                        &mapped, cap, ws, ws_bytes, stream);
}

int shc_compact_mask_table_start(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                                 int32_t* inv, int32_t* row_ptr, int32_t* n_active_dev,
                                 int64_t* n_active_host, int64_t cap, const int32_t* nbr,
                                 int32_t K, int32_t* table, void* ws, size_t ws_bytes,
                                 hipStream_t stream) {
  g_last_error[0] = 0;
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  if (V > shc::kCompactTableMaxV)
    return fail(SHC_ERR_UNSUPPORTED, "V = %d exceeds the %d vertices of a body this call keeps",
                V, shc::kCompactTableMaxV);
  SHC_PTR(nbr, "nbr");
  if (cap > 0) SHC_PTR(table, "table");
  int64_t* mapped = nullptr;
  return compact_launch(mask, B, V, coords, inv, row_ptr, n_active_dev, n_active_host, true,
                        &mapped, cap, ws, ws_bytes, stream, nbr, K, cap > 0 ? table : nullptr);
}

int shc_compact_mask_wait(int64_t* n_active_host, int64_t cap, hipStream_t stream) {
  g_last_error[0] = 0;
  if (n_active_host == nullptr) return fail(SHC_ERR_INVALID_ARG, "n_active_host is NULL");
  // The compaction stores N' into the page-locked variable as soon as it is
  // known; poll it rather than waiting for the whole stream (later work on
  // the stream is ordered after the compaction anyway).  Every few thousand
  // polls the stream is queried, so a failed launch or a stream that drains
  // without a count ends the wait.
  volatile int64_t* host_count = n_active_host;
  int64_t n = 0;
  for (uint64_t it = 1;; ++it) {
    n = *host_count;
    if (n >= 0) break;
    if ((it & 4095u) == 0) {
      const hipError_t q = hipStreamQuery(stream);
      if (q == hipSuccess) {
        n = *host_count;
        if (n < 0) return fail(SHC_ERR_HIP, "compact_mask: stream finished without a count");
        break;
      }
      if (q != hipErrorNotReady) return hip_status(q, "compact_mask stream query");
    }
  }
  if (n > cap)
    return fail(SHC_ERR_CAPACITY, "N' = %lld active rows exceed cap = %lld", (long long)n,
                (long long)cap);
  return SHC_OK;
}

int shc_compact_mask(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords, int32_t* inv,
                     int32_t* row_ptr, int32_t* n_active_dev, int64_t* n_active_host, int64_t cap,
                     void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  int64_t* mapped = nullptr;
  int rc = compact_launch(mask, B, V, coords, inv, row_ptr, n_active_dev, n_active_host, false,
                          &mapped, cap, ws, ws_bytes, stream);
  if (rc != SHC_OK || n_active_host == nullptr) return rc;
  if (mapped != nullptr) return shc_compact_mask_wait(n_active_host, cap, stream);
  // pageable host memory: a copy and a full stream synchronisation
  int32_t n32 = 0;
  rc = hip_status(hipMemcpyAsync(&n32, n_active_dev, sizeof(int32_t), hipMemcpyDeviceToHost, stream),
                  "compact_mask count copy");
  if (rc != SHC_OK) return rc;
  rc = hip_status(hipStreamSynchronize(stream), "compact_mask stream sync");
  if (rc != SHC_OK) return rc;
  *n_active_host = n32;
  if (n32 > cap)
    return fail(SHC_ERR_CAPACITY, "N' = %lld active rows exceed cap = %lld", (long long)n32,
                (long long)cap);
  return SHC_OK;
}

}  // extern "C"

// Scratch of shc_compact_mask_noalloc: the compaction's per-span counts, in
// device memory the library owns instead of a caller's workspace.  Every GPU
// the library runs on holds its own copy of the array until the process
// ends.  Host code never passes the array's name to a kernel (on the host it
// names a stand-in, not the device copy): scratch_address() resolves the
// current device's copy once and every use goes through that pointer.
static constexpr size_t kNoAllocScratchBytes = 64 * 1024;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices];  // device copy of `scratch`, per device

// Device address of the current device's `scratch`, resolved on the first
// call on that device (with the device current) and kept.
int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_status(e, "compact_mask_noalloc device query");
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(SHC_ERR_UNSUPPORTED, "device %d is beyond the %d this library serves", dev,
                kMaxScratchDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_status(e, "compact_mask_noalloc scratch address");
    if (p == nullptr) return fail(SHC_ERR_HIP, "compact_mask_noalloc: scratch address is NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SHC_OK;
}

}  // namespace

extern "C" {

int shc_compact_mask_noalloc(const uint8_t* mask, int32_t B, int32_t V, int32_t* coords,
                             int32_t* inv, int32_t* row_ptr, int32_t* n_active_dev,
                             int64_t* n_active_host, int64_t cap, hipStream_t stream) {
  g_last_error[0] = 0;
  // the arguments are checked before the scratch address is looked up, so
  // a bad call touches no device
  SHC_TRY(check_bv(B, V));
  SHC_PTR(mask, "mask");
  SHC_PTR(inv, "inv");
  SHC_PTR(row_ptr, "row_ptr");
  SHC_PTR(n_active_dev, "n_active_dev");
  if (cap < 0) return fail(SHC_ERR_INVALID_ARG, "cap = %lld is negative", (long long)cap);
  if (cap > 0) SHC_PTR(coords, "coords");
  const size_t need = shc_compact_mask_workspace(B, V);
  if (need > kNoAllocScratchBytes)
    return fail(SHC_ERR_CAPACITY, "a %d x %d mask needs %zu bytes of scratch, above the %zu "
                "this call holds", B, V, need, kNoAllocScratchBytes);
  void* ws = nullptr;
  SHC_TRY(scratch_address(&ws));
  return shc_compact_mask(mask, B, V, coords, inv, row_ptr, n_active_dev, n_active_host, cap, ws,
                          kNoAllocScratchBytes, stream);
}

int shc_gather_rows(const void* x, const int32_t* coords, int64_t n_rows, int32_t B, int32_t V,
                    int32_t C, int32_t dtype, void* S, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(x, "x");
  SHC_PTR(coords, "coords");
  SHC_PTR(S, "S");
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(shc::launch_gather(x, coords, n_rows, B, V, row_bytes, S, stream),
                    "gather_rows launch");
}

int shc_gather_rows_stacked(const void* x, const int32_t* coords, int64_t n_rows, int32_t B,
                            int32_t kappa, int32_t V, int32_t C, int32_t dtype, void* S,
                            hipStream_t stream) {
  g_last_error[0] = 0;
  if (kappa <= 0) return fail(SHC_ERR_INVALID_ARG, "kappa = %d must be positive", kappa);
  if ((int64_t)kappa * B > 0x7FFFFFFFLL)
    return fail(SHC_ERR_UNSUPPORTED, "kappa * B = %lld bodies exceed int32", (long long)kappa * B);
  SHC_TRY(check_bv(kappa * B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(x, "x");
  SHC_PTR(coords, "coords");
  SHC_PTR(S, "S");
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(shc::launch_gather_ext(x, nullptr, 0, coords, n_rows, kappa * B, B, V,
                                           row_bytes, S, stream),
                    "gather_rows_stacked launch");
}

int shc_gather_rows_masked(const void* x, const uint8_t* me, const int32_t* coords,
                           int64_t n_rows, int32_t B, int32_t V, int32_t C, int32_t dtype,
                           void* S, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(x, "x");
  SHC_PTR(me, "me");
  SHC_PTR(coords, "coords");
  SHC_PTR(S, "S");
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(shc::launch_gather_ext(x, me, dtype == SHC_BF16 ? 1 : 2, coords, n_rows, B, B,
                                           V, row_bytes, S, stream),
                    "gather_rows_masked launch");
}

int shc_row_mask_from_elements(const uint8_t* me, int32_t B, int32_t V, int32_t C, uint8_t* m,
                               hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_channels("C", C));
  SHC_PTR(me, "me");
  SHC_PTR(m, "m");
  return hip_status(shc::launch_row_activity(me, B, V, C, m, stream),
                    "row_mask_from_elements launch");
}

int shc_combine_stacked(const void* Y, int32_t kappa, int64_t rows, int32_t C, int32_t dtype,
                        int32_t op, void* out, hipStream_t stream) {
  g_last_error[0] = 0;
  if (kappa <= 0) return fail(SHC_ERR_INVALID_ARG, "kappa = %d must be positive", kappa);
  SHC_TRY(check_rows(rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (op != SHC_COMBINE_SUM && op != SHC_COMBINE_MEAN && op != SHC_COMBINE_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "unknown combination code %d", op);
  if (rows == 0) return SHC_OK;
  SHC_PTR(Y, "Y");
  SHC_PTR(out, "out");
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(shc::launch_combine(Y, kappa, rows, row_bytes, op, dtype == SHC_BF16, out,
                                        stream),
                    "combine_stacked launch");
}

int shc_sparse_linear(const void* S, int64_t n_rows, const void* W, const float* bias, int32_t Cin,
                      int32_t Cout, int32_t dtype, int32_t act, void* out, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("Cin", Cin));
  SHC_TRY(check_channels("Cout", Cout));
  if (act != SHC_ACT_NONE && act != SHC_ACT_RELU)
    return fail(SHC_ERR_UNSUPPORTED, "unknown activation code %d", act);
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(W, "W");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  shc::GemmArgs a{};
  a.S = S;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.B = 1;
  a.V = 1;
  a.K = 1;
  a.Cin = Cin;
  a.Cout = Cout;
  a.relu = act == SHC_ACT_RELU;
  return hip_status(shc::launch_gather_gemm(a, false, dtype == SHC_BF16, stream),
                    "sparse_linear launch");
}

int shc_gather_sparse_linear(const void* x, const int32_t* coords, int64_t n_rows, int32_t B,
                             int32_t V, const void* W, const float* bias, int32_t Cin,
                             int32_t Cout, int32_t dtype, int32_t act, void* out,
                             hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("Cin", Cin));
  SHC_TRY(check_channels("Cout", Cout));
  if (act != SHC_ACT_NONE && act != SHC_ACT_RELU)
    return fail(SHC_ERR_UNSUPPORTED, "unknown activation code %d", act);
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(x, "x");
  SHC_PTR(coords, "coords");
  SHC_PTR(W, "W");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  shc::GemmArgs a{};
  a.S = x;
  a.coords = coords;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.B = B;
  a.V = V;
  a.K = 1;
  a.Cin = Cin;
  a.Cout = Cout;
  a.relu = act == SHC_ACT_RELU;
  a.gather = 1;
  return hip_status(shc::launch_gather_gemm(a, false, dtype == SHC_BF16, stream),
                    "gather_sparse_linear launch");
}

int shc_sparse_neighbor_conv(const void* S, const int32_t* coords, const int32_t* inv,
                             int64_t n_rows, int32_t B, int32_t V, const int32_t* nbr, int32_t K,
                             const void* W, const float* bias, int32_t Cin, int32_t Cout,
                             int32_t dtype, int32_t act, void* out, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("Cin", Cin));
  SHC_TRY(check_channels("Cout", Cout));
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  if (act != SHC_ACT_NONE && act != SHC_ACT_RELU)
    return fail(SHC_ERR_UNSUPPORTED, "unknown activation code %d", act);
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(coords, "coords");
  SHC_PTR(inv, "inv");
  SHC_PTR(nbr, "nbr");
  SHC_PTR(W, "W");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  shc::GemmArgs a{};
  a.S = S;
  a.coords = coords;
  a.inv = inv;
  a.nbr = nbr;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.B = B;
  a.V = V;
  a.K = K;
  a.Cin = Cin;
  a.Cout = Cout;
  a.relu = act == SHC_ACT_RELU;
  return hip_status(shc::launch_gather_gemm(a, true, dtype == SHC_BF16, stream),
                    "sparse_neighbor_conv launch");
}

int shc_build_neighbor_table(const int32_t* coords, const int32_t* inv, int64_t n_rows,
                             int32_t B, int32_t V, const int32_t* nbr, int32_t K, int32_t* table,
                             hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(coords, "coords");
  SHC_PTR(inv, "inv");
  SHC_PTR(nbr, "nbr");
  SHC_PTR(table, "table");
  return hip_status(shc::launch_neighbor_table(coords, inv, n_rows, B, V, nbr, K, table, stream),
                    "build_neighbor_table launch");
}

}  // extern "C"

namespace {

// Shape checks shared by the table conv, its plan and the planned conv.
int check_conv_shape(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype,
                     int32_t act) {
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("Cin", Cin));
  SHC_TRY(check_channels("Cout", Cout));
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  if (act != SHC_ACT_NONE && act != SHC_ACT_RELU)
    return fail(SHC_ERR_UNSUPPORTED, "unknown activation code %d", act);
  return SHC_OK;
}

// A conv shape on the current device for the plan queries (false: no device).
bool plan_shape(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, shc::GemmArgs* a,
                int* cus) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return false;
  *a = shc::GemmArgs{};
  a->n_rows = n_rows;
  a->B = 1;
  a->V = 1;
  a->K = K;
  a->Cin = Cin;
  a->Cout = Cout;
  return true;
}

// Plan size and row-group stride of a conv of exactly n_rows rows (0: no
// plan for this shape, or no device).
int64_t plan_size(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype,
                  int64_t* stride) {
  *stride = 0;
  shc::GemmArgs a{};
  int cus = 0;
  if (!plan_shape(n_rows, K, Cin, Cout, &a, &cus)) return 0;
  return shc::conv_plan_bytes(a, dtype == SHC_BF16, cus, stride);
}

bool plan_query_args_ok(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype) {
  return n_rows > 0 && n_rows <= INT32_MAX && K > 0 && K <= kMaxSlots && Cin > 0 &&
         Cin % 16 == 0 && Cin <= kMaxChannels && Cout > 0 && Cout % 16 == 0 &&
         Cout <= kMaxChannels && (dtype == SHC_F32 || dtype == SHC_BF16);
}

// The plan buffer of a build or planned call: present, and large enough for
// this shape's plan.
int check_plan(const void* plan, size_t plan_bytes, int64_t n_rows, int32_t K, int32_t Cin,
               int32_t Cout, int32_t dtype, int64_t* stride) {
  SHC_PTR(plan, "plan");
  const int64_t need = plan_size(n_rows, K, Cin, Cout, dtype, stride);
  if (need == 0)
    return fail(SHC_ERR_UNSUPPORTED,
                "no conv plan for n_rows = %lld, K = %d, Cin = %d, Cout = %d, dtype %d on "
                "this device",
                (long long)n_rows, K, Cin, Cout, dtype);
  if ((int64_t)plan_bytes < need)
    return fail(SHC_ERR_CAPACITY, "plan_bytes = %zu is below the %lld bytes of this plan",
                plan_bytes, (long long)need);
  return SHC_OK;
}

}  // namespace

extern "C" {

int shc_sparse_neighbor_conv_table(const void* S, const int32_t* table, int64_t n_rows,
                                   int32_t K, const void* W, const float* bias, int32_t Cin,
                                   int32_t Cout, int32_t dtype, int32_t act, void* out,
                                   hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_conv_shape(n_rows, K, Cin, Cout, dtype, act));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(table, "table");
  SHC_PTR(W, "W");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  shc::GemmArgs a{};
  a.S = S;
  a.table = table;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.B = 1;
  a.V = 1;
  a.K = K;
  a.Cin = Cin;
  a.Cout = Cout;
  a.relu = act == SHC_ACT_RELU;
  return hip_status(shc::launch_gather_gemm(a, true, dtype == SHC_BF16, stream),
                    "sparse_neighbor_conv_table launch");
}

size_t shc_conv_split_workspace_bytes(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout,
                                      int32_t dtype) {
  if (n_rows < 0 || n_rows > INT32_MAX || dtype != SHC_BF16 ||
      !shc::conv_split_supported(n_rows, K, Cin, Cout))
    return 0;
  const int64_t b = shc::conv_split_workspace_bytes(n_rows, K, Cout);
  return (size_t)(b > 16 ? b : 16);
}

int shc_sparse_neighbor_conv_split(const void* S, const int32_t* table, int64_t n_rows,
                                   int32_t K, const void* W, const float* bias, int32_t Cin,
                                   int32_t Cout, int32_t dtype, int32_t act, void* out,
                                   void* workspace, size_t workspace_bytes,
                                   hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_conv_shape(n_rows, K, Cin, Cout, dtype, act));
  if (dtype != SHC_BF16)
    return fail(SHC_ERR_UNSUPPORTED, "the split conv runs bf16 only (dtype %d)", dtype);
  if (!shc::conv_split_supported(n_rows, K, Cin, Cout))
    return fail(SHC_ERR_UNSUPPORTED,
                "no split conv for n_rows = %lld, K = %d, Cin = %d, Cout = %d (channels in "
                "{64, 128, 256}, (K - 1) * n_rows * Cout * 4 below 2^31)",
                (long long)n_rows, K, Cin, Cout);
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(table, "table");
  SHC_PTR(W, "W");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  SHC_PTR(workspace, "workspace");
  const int64_t need = shc::conv_split_workspace_bytes(n_rows, K, Cout);
  if ((int64_t)workspace_bytes < need)
    return fail(SHC_ERR_CAPACITY, "workspace_bytes = %zu is below the %lld bytes this call needs",
                workspace_bytes, (long long)need);
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_status(e, "sparse_neighbor_conv_split device query");
  return hip_status(shc::launch_conv_split(S, table, n_rows, K, W, bias, Cin, Cout,
                                           act == SHC_ACT_RELU, out,
                                           static_cast<float*>(workspace), cus, stream),
                    "sparse_neighbor_conv_split launch");
}

size_t shc_conv_packed_weights_bytes(int32_t K, int32_t Cin, int32_t Cout, int32_t dtype) {
  if (dtype != SHC_BF16 || !shc::conv_packed_supported(1, K, Cin, Cout)) return 0;
  return (size_t)shc::conv_packed_weights_bytes(K, Cin, Cout);
}

int shc_pack_conv_weights(const void* W, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype,
                          void* Wp, size_t Wp_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_conv_shape(1, K, Cin, Cout, dtype, SHC_ACT_NONE));
  if (dtype != SHC_BF16 || !shc::conv_packed_supported(1, K, Cin, Cout))
    return fail(SHC_ERR_UNSUPPORTED,
                "no packed conv for dtype %d, K = %d, Cin = %d, Cout = %d (bf16, K <= 9, "
                "channels in {64, 128})",
                dtype, K, Cin, Cout);
  SHC_PTR(W, "W");
  SHC_PTR(Wp, "Wp");
  const int64_t need = shc::conv_packed_weights_bytes(K, Cin, Cout);
  if ((int64_t)Wp_bytes < need)
    return fail(SHC_ERR_CAPACITY, "Wp_bytes = %zu is below the %lld bytes of the packed weights",
                Wp_bytes, (long long)need);
  return hip_status(shc::launch_pack_conv_weights(W, K, Cin, Cout, Wp, stream),
                    "pack_conv_weights launch");
}

int shc_sparse_neighbor_conv_packed(const void* S, const int32_t* table, int64_t n_rows,
                                    int32_t K, const void* Wp, const float* bias, int32_t Cin,
                                    int32_t Cout, int32_t dtype, int32_t act, void* out,
                                    hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_conv_shape(n_rows, K, Cin, Cout, dtype, act));
  if (dtype != SHC_BF16 || !shc::conv_packed_supported(n_rows, K, Cin, Cout))
    return fail(SHC_ERR_UNSUPPORTED,
                "no packed conv for dtype %d, K = %d, Cin = %d, Cout = %d (bf16, K <= 9, "
                "channels in {64, 128})",
                dtype, K, Cin, Cout);
  // the table is read through a buffer resource of K * n_rows * 4 bytes
  if ((int64_t)K * n_rows * 4 > 0x7FFFFFFFLL)
    return fail(SHC_ERR_UNSUPPORTED, "K * n_rows * 4 = %lld bytes of table exceed 2^31 - 1",
                (long long)((int64_t)K * n_rows * 4));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(table, "table");
  SHC_PTR(Wp, "Wp");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_status(e, "sparse_neighbor_conv_packed device query");
  return hip_status(shc::launch_conv_packed(S, table, n_rows, K, Wp, bias, Cin, Cout,
                                            act == SHC_ACT_RELU, out, cus, stream),
                    "sparse_neighbor_conv_packed launch");
}

namespace {
int device_cus(int* cus) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(cus, hipDeviceAttributeMultiprocessorCount, dev);
  return e == hipSuccess ? SHC_OK : hip_status(e, "device query");
}

int check_packed_shape(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype,
                       int32_t act) {
  SHC_TRY(check_conv_shape(n_rows, K, Cin, Cout, dtype, act));
  if (dtype != SHC_BF16 || !shc::conv_packed_supported(n_rows, K, Cin, Cout))
    return fail(SHC_ERR_UNSUPPORTED,
                "no packed conv for dtype %d, K = %d, Cin = %d, Cout = %d (bf16, K <= 9, "
                "channels in {64, 128})",
                dtype, K, Cin, Cout);
  if ((int64_t)K * n_rows * 4 > 0x7FFFFFFFLL)
    return fail(SHC_ERR_UNSUPPORTED, "K * n_rows * 4 = %lld bytes of table exceed 2^31 - 1",
                (long long)((int64_t)K * n_rows * 4));
  return SHC_OK;
}
}  // namespace

size_t shc_conv_packed_plan_bytes(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout,
                                  int32_t dtype) {
  if (n_rows < 0 || dtype != SHC_BF16 || !shc::conv_packed_supported(n_rows, K, Cin, Cout) ||
      (int64_t)K * n_rows * 4 > 0x7FFFFFFFLL)
    return 0;
  int cus = 0;
  if (device_cus(&cus) != SHC_OK) return 0;
  const int64_t b = shc::conv_packed_plan_bytes_upto(n_rows, Cin, Cout, cus);
  return (size_t)(b > 16 ? b : 16);
}

int shc_build_conv_packed_plan(const int32_t* table, int64_t n_rows, int32_t K, int32_t Cin,
                               int32_t Cout, int32_t dtype, void* plan, size_t plan_bytes,
                               hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_packed_shape(n_rows, K, Cin, Cout, dtype, SHC_ACT_NONE));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(table, "table");
  SHC_PTR(plan, "plan");
  int cus = 0;
  SHC_TRY(device_cus(&cus));
  const int64_t need = shc::conv_packed_plan_bytes(n_rows, Cin, Cout, cus);
  if ((int64_t)plan_bytes < need)
    return fail(SHC_ERR_CAPACITY, "plan_bytes = %zu is below the %lld bytes of this plan",
                plan_bytes, (long long)need);
  return hip_status(shc::launch_build_packed_plan(table, n_rows, K, Cin, Cout, plan, cus, stream),
                    "build_conv_packed_plan launch");
}

int shc_sparse_neighbor_conv_packed_planned(const void* S, const void* plan, size_t plan_bytes,
                                            int64_t n_rows, int32_t K, const void* Wp,
                                            const float* bias, int32_t Cin, int32_t Cout,
                                            int32_t dtype, int32_t act, void* out,
                                            hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_packed_shape(n_rows, K, Cin, Cout, dtype, act));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(plan, "plan");
  SHC_PTR(Wp, "Wp");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  int cus = 0;
  SHC_TRY(device_cus(&cus));
  const int64_t need = shc::conv_packed_plan_bytes(n_rows, Cin, Cout, cus);
  if ((int64_t)plan_bytes < need)
    return fail(SHC_ERR_CAPACITY, "plan_bytes = %zu is below the %lld bytes of a plan of "
                "%lld rows", plan_bytes, (long long)need, (long long)n_rows);
  return hip_status(shc::launch_conv_packed_planned(S, plan, n_rows, K, Wp, bias, Cin, Cout,
                                                    act == SHC_ACT_RELU, out, cus, stream),
                    "sparse_neighbor_conv_packed_planned launch");
}

size_t shc_conv_plan_bytes(int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout, int32_t dtype) {
  if (!plan_query_args_ok(n_rows, K, Cin, Cout, dtype)) return 0;
  shc::GemmArgs a{};
  int cus = 0;
  if (!plan_shape(n_rows, K, Cin, Cout, &a, &cus)) return 0;
  return (size_t)shc::conv_plan_bytes_upto(a, dtype == SHC_BF16, cus);
}

int64_t shc_conv_plan_max_rows(int32_t K, int32_t Cin, int32_t Cout, int32_t dtype) {
  if (!plan_query_args_ok(1, K, Cin, Cout, dtype)) return 0;
  shc::GemmArgs a{};
  int cus = 0;
  if (!plan_shape(1, K, Cin, Cout, &a, &cus)) return 0;
  return shc::conv_plan_max_rows(a, dtype == SHC_BF16, cus);
}

int shc_build_conv_plan(const int32_t* table, int64_t n_rows, int32_t K, int32_t Cin,
                        int32_t Cout, int32_t dtype, void* plan, size_t plan_bytes,
                        hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_conv_shape(n_rows, K, Cin, Cout, dtype, SHC_ACT_NONE));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(table, "table");
  int64_t stride;
  SHC_TRY(check_plan(plan, plan_bytes, n_rows, K, Cin, Cout, dtype, &stride));
  shc::GemmArgs a{};
  a.table = table;
  a.n_rows = n_rows;
  a.B = 1;
  a.V = 1;
  a.K = K;
  a.Cin = Cin;
  a.Cout = Cout;
  a.plan_out = plan;
  a.plan_stride = stride;
  return hip_status(shc::launch_gather_gemm(a, true, dtype == SHC_BF16, stream),
                    "build_conv_plan launch");
}

int shc_sparse_neighbor_conv_planned(const void* S, const void* plan, size_t plan_bytes,
                                     int64_t n_rows, int32_t K, const void* W,
                                     const float* bias, int32_t Cin, int32_t Cout,
                                     int32_t dtype, int32_t act, void* out,
                                     hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_conv_shape(n_rows, K, Cin, Cout, dtype, act));
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(W, "W");
  SHC_OPT_PTR(bias, "bias");
  SHC_PTR(out, "out");
  int64_t stride;
  SHC_TRY(check_plan(plan, plan_bytes, n_rows, K, Cin, Cout, dtype, &stride));
  shc::GemmArgs a{};
  a.S = S;
  a.W = W;
  a.bias = bias;
  a.out = out;
  a.n_rows = n_rows;
  a.B = 1;
  a.V = 1;
  a.K = K;
  a.Cin = Cin;
  a.Cout = Cout;
  a.relu = act == SHC_ACT_RELU;
  a.plan = plan;
  a.plan_stride = stride;
  return hip_status(shc::launch_gather_gemm(a, true, dtype == SHC_BF16, stream),
                    "sparse_neighbor_conv_planned launch");
}

int shc_scatter(const void* S, const int32_t* inv, const int32_t* coords, int64_t n_rows,
                int32_t B, int32_t V, int32_t C, int32_t dtype, int32_t zero_fill, void* D,
                hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (zero_fill != 0 && zero_fill != 1)
    return fail(SHC_ERR_INVALID_ARG, "zero_fill = %d must be 0 or 1", zero_fill);
  SHC_PTR(D, "D");
  if (zero_fill) {
    SHC_PTR(inv, "inv");
    if (n_rows > 0) SHC_PTR(S, "S");
  } else {
    if (n_rows == 0) return SHC_OK;
    SHC_PTR(coords, "coords");
    SHC_PTR(S, "S");
  }
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(
      shc::launch_scatter(S, inv, coords, n_rows, B, V, row_bytes, zero_fill, D, stream),
      "scatter launch");
}

int shc_scatter_update(const void* S, const int32_t* inv, const int32_t* coords, int64_t n_rows,
                       const int32_t* prev_coords, int64_t prev_rows, int32_t B, int32_t V,
                       int32_t C, int32_t dtype, void* D, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_rows(prev_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (n_rows + prev_rows == 0) return SHC_OK;
  SHC_PTR(D, "D");
  SHC_PTR(inv, "inv");
  if (n_rows > 0) {
    SHC_PTR(S, "S");
    SHC_PTR(coords, "coords");
  }
  if (prev_rows > 0) SHC_PTR(prev_coords, "prev_coords");
  if (prev_coords != nullptr && prev_coords == coords)
    return fail(SHC_ERR_INVALID_ARG, "prev_coords and coords are the same buffer");
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(shc::launch_scatter_update(S, inv, coords, n_rows, prev_coords, prev_rows, B,
                                               V, row_bytes, D, stream),
                    "scatter_update launch");
}

int shc_clear_inactive_rows(const int32_t* inv, int32_t B, int32_t V, int32_t C, int32_t dtype,
                            void* D, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  SHC_PTR(inv, "inv");
  SHC_PTR(D, "D");
  const int32_t row_bytes = C * (dtype == SHC_BF16 ? 2 : 4);
  return hip_status(shc::launch_clear_inactive(inv, B, V, row_bytes, D, stream),
                    "clear_inactive_rows launch");
}

int shc_segment_group_norm(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                           int32_t C, int32_t G, float eps, int32_t dtype, void* out,
                           hipStream_t stream) {
  g_last_error[0] = 0;
  if (B <= 0) return fail(SHC_ERR_INVALID_ARG, "B = %d must be positive", B);
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  if (G <= 0 || C % G != 0)
    return fail(SHC_ERR_INVALID_ARG, "G = %d must be positive and divide C = %d", G, C);
  if (!(eps > 0.f) || !std::isfinite(eps))
    return fail(SHC_ERR_INVALID_ARG, "eps = %g must be positive and finite", (double)eps);
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(S, "S");
  SHC_PTR(row_ptr, "row_ptr");
  SHC_PTR(out, "out");
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_status(e, "segment_group_norm device query");
  return hip_status(shc::launch_group_norm(S, row_ptr, n_rows, B, C, G, eps, dtype == SHC_BF16,
                                           out, cus, stream),
                    "segment_group_norm launch");
}

size_t shc_mask_scores_workspace(int32_t K, int64_t N, int32_t C) {
  if (K < 1 || K > shc::kMaxScoreMasks || N < 0 || C < 64 || C > 1024 || C % 64 != 0) return 0;
  return shc::mask_scores_workspace_bytes(K, N, C);
}

int shc_mask_scores(const void* O, int32_t K, int64_t N, int32_t C, int32_t dtype,
                    const double* alpha_in, double* alpha_out, double* sim, int32_t kappa,
                    int32_t* top, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  if (K < 1 || K > shc::kMaxScoreMasks)
    return fail(SHC_ERR_UNSUPPORTED, "K = %d masks outside [1, %d]", K, shc::kMaxScoreMasks);
  if (N < 1) return fail(SHC_ERR_INVALID_ARG, "N = %lld rows must be positive", (long long)N);
  if (dtype != SHC_BF16) return fail(SHC_ERR_UNSUPPORTED, "mask scores take bf16 outputs");
  if (C < 64 || C > 1024 || C % 64 != 0)
    return fail(SHC_ERR_UNSUPPORTED, "C = %d must be a multiple of 64 in [64, 1024]", C);
  if (kappa < 0 || kappa > K)
    return fail(SHC_ERR_INVALID_ARG, "kappa = %d outside [0, K = %d]", kappa, K);
  SHC_PTR(O, "O");
  SHC_PTR(alpha_out, "alpha_out");
  SHC_OPT_PTR(alpha_in, "alpha_in");
  SHC_OPT_PTR(sim, "sim");
  SHC_OPT_PTR(top, "top");
  if (kappa > 0 && top == nullptr) return fail(SHC_ERR_INVALID_ARG, "kappa > 0 needs top");
  SHC_PTR(ws, "ws");
  const size_t need = shc_mask_scores_workspace(K, N, C);
  if (ws_bytes < need)
    return fail(SHC_ERR_CAPACITY, "workspace of %zu bytes is below the %zu needed", ws_bytes, need);
  return hip_status(shc::launch_mask_scores(O, K, N, C, alpha_in, alpha_out, sim, kappa, top, ws,
                                            stream),
                    "mask_scores launch");
}

size_t shc_transpose_neighbors_workspace(int32_t V, int32_t K) {
  if (V <= 0 || K <= 0 || K > kMaxSlots) return 0;
  return shc::transpose_neighbors_ws_bytes(V, K);
}

int shc_transpose_neighbors(const int32_t* nbr, int32_t V, int32_t K, int32_t* nbr_t,
                            int32_t* slot_of, int32_t* Kt_host, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  g_last_error[0] = 0;
  if (V <= 0) return fail(SHC_ERR_INVALID_ARG, "V = %d must be positive", V);
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  if ((int64_t)V * SHC_MAX_VIRTUAL_SLOTS > INT32_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "V = %d is too large for the transposed lists", V);
  SHC_PTR(nbr, "nbr");
  SHC_PTR(nbr_t, "nbr_t");
  SHC_PTR(slot_of, "slot_of");
  SHC_PTR(ws, "ws");
  if (Kt_host == nullptr) return fail(SHC_ERR_INVALID_ARG, "Kt_host is NULL");
  const size_t need = shc_transpose_neighbors_workspace(V, K);
  if (ws_bytes < need)
    return fail(SHC_ERR_CAPACITY, "workspace of %zu bytes is below the %zu needed", ws_bytes, need);
  // the slot offsets follow the two count arrays in the workspace
  int32_t* off = reinterpret_cast<int32_t*>(static_cast<unsigned char*>(ws) + need -
                                            (((size_t)(K + 1) * 4 + 255) & ~(size_t)255));
  SHC_TRY(hip_status(shc::launch_transpose_neighbors(nbr, V, K, nbr_t, slot_of, off, ws, stream),
                     "transpose_neighbors launch"));
  int32_t kt = 0;
  SHC_TRY(hip_status(hipMemcpyAsync(&kt, off + K, sizeof(int32_t), hipMemcpyDeviceToHost, stream),
                     "transpose_neighbors Kt copy"));
  SHC_TRY(hip_status(hipStreamSynchronize(stream), "transpose_neighbors stream sync"));
  *Kt_host = kt;
  if (kt > SHC_MAX_VIRTUAL_SLOTS)
    return fail(SHC_ERR_UNSUPPORTED, "the mesh needs Kt = %d virtual slots, above %d", kt,
                SHC_MAX_VIRTUAL_SLOTS);
  return SHC_OK;
}

int shc_build_transposed_table(const int32_t* coords, const int32_t* inv, int64_t n_rows,
                               int32_t B, int32_t V, const int32_t* nbr_t, int32_t Kt,
                               int32_t* table_t, uint64_t* row_slots, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_bv(B, V));
  SHC_TRY(check_rows(n_rows));
  if (Kt < 1 || Kt > SHC_MAX_VIRTUAL_SLOTS)
    return fail(SHC_ERR_INVALID_ARG, "Kt = %d outside [1, %d]", Kt, SHC_MAX_VIRTUAL_SLOTS);
  if ((int64_t)Kt * n_rows > INT32_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "Kt * n_rows exceeds 2^31 - 1");
  if (n_rows == 0) return SHC_OK;
  SHC_PTR(coords, "coords");
  SHC_PTR(inv, "inv");
  SHC_PTR(nbr_t, "nbr_t");
  SHC_PTR(table_t, "table_t");
  SHC_PTR(row_slots, "row_slots");
  return hip_status(shc::launch_transposed_table(coords, inv, n_rows, B, V, nbr_t, Kt, table_t,
                                                 row_slots, stream),
                    "build_transposed_table launch");
}

// Shared checks of the two layer backward calls.
static int check_backward(const void* S, const void* W, const void* Y, const void* dY,
                          int64_t n_rows, int32_t Kw, int32_t Cin, int32_t Cout, int32_t dtype,
                          int32_t act, const void* dS, const float* dW, const float* db,
                          const void* ws, size_t ws_bytes, size_t need) {
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("Cin", Cin));
  SHC_TRY(check_channels("Cout", Cout));
  if (Cout > 256) return fail(SHC_ERR_UNSUPPORTED, "Cout = %d above 256", Cout);
  if (act != SHC_ACT_NONE && act != SHC_ACT_RELU)
    return fail(SHC_ERR_UNSUPPORTED, "unknown activation code %d", act);
  const int64_t e = dtype == SHC_BF16 ? 2 : 4;
  if (n_rows * (int64_t)(Cin > Cout ? Cin : Cout) * e > INT32_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "a feature tensor of %lld rows exceeds 2 GiB",
                (long long)n_rows);
  if (dS != nullptr && !shc::backward_dgrad_supported(Kw, Cin, Cout, dtype == SHC_BF16))
    return fail(SHC_ERR_UNSUPPORTED, "input gradient for K = %d, Cin = %d, Cout = %d does not fit",
                Kw, Cin, Cout);
  SHC_OPT_PTR(dS, "dS");
  SHC_OPT_PTR(dW, "dW");
  SHC_OPT_PTR(db, "db");
  if (n_rows > 0) {
    SHC_PTR(dY, "dY");
    if (act == SHC_ACT_RELU) SHC_PTR(Y, "Y");
    if (dW != nullptr) SHC_PTR(S, "S");
  }
  if (dS != nullptr || dW != nullptr) SHC_PTR(W, "W");
  if (n_rows > 0 || dW != nullptr || db != nullptr) SHC_PTR(ws, "ws");
  if (ws_bytes < need)
    return fail(SHC_ERR_CAPACITY, "workspace of %zu bytes is below the %zu needed", ws_bytes, need);
  return SHC_OK;
}

size_t shc_sparse_linear_backward_workspace(int64_t n_rows, int32_t Cin, int32_t Cout,
                                            int32_t dtype) {
  if (n_rows < 0 || Cin <= 0 || Cout <= 0 || (dtype != SHC_BF16 && dtype != SHC_F32)) return 0;
  shc::BwdPlan pl;
  shc::backward_plan(n_rows, 1, Cin, Cout, dtype == SHC_BF16, 0, &pl);
  return pl.total;
}

int shc_sparse_linear_backward(const void* S, const void* W, const void* Y, const void* dY,
                               int64_t n_rows, int32_t Cin, int32_t Cout, int32_t dtype,
                               int32_t act, void* dS, float* dW, float* db, void* ws,
                               size_t ws_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_backward(S, W, Y, dY, n_rows, 1, Cin, Cout, dtype, act, dS, dW, db, ws, ws_bytes,
                         shc_sparse_linear_backward_workspace(n_rows, Cin, Cout, dtype)));
  return hip_status(shc::launch_layer_backward(0, S, nullptr, nullptr, nullptr, nullptr, nullptr,
                                               nullptr, W, Y, dY, n_rows, 1, Cin, Cout,
                                               dtype == SHC_BF16, act, dS, dW, db, ws, stream),
                    "sparse_linear_backward launch");
}

size_t shc_sparse_neighbor_conv_backward_workspace(int64_t n_rows, int32_t K, int32_t Cin,
                                                   int32_t Cout, int32_t dtype) {
  if (n_rows < 0 || K <= 0 || K > kMaxSlots || Cin <= 0 || Cout <= 0 ||
      (dtype != SHC_BF16 && dtype != SHC_F32))
    return 0;
  shc::BwdPlan pl;
  shc::backward_plan(n_rows, K, Cin, Cout, dtype == SHC_BF16, 1, &pl);
  return pl.total;
}

size_t shc_build_slot_pairs_workspace(int64_t n_rows, int32_t K) {
  if (n_rows < 0 || K <= 0 || K > kMaxSlots) return 0;
  return shc::slot_pairs_ws_bytes(n_rows, K);
}

int shc_build_slot_pairs(const int32_t* table, int64_t n_rows, int32_t K, int32_t* pairs,
                         int32_t* pair_ptr, void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  SHC_TRY(check_rows(n_rows));
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  if ((int64_t)K * n_rows > INT32_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "K * n_rows exceeds 2^31 - 1");
  SHC_PTR(pair_ptr, "pair_ptr");
  if (n_rows == 0)
    return hip_status(shc::launch_fill_i32(pair_ptr, K + 1, 0, stream),
                      "build_slot_pairs empty offsets");
  SHC_PTR(table, "table");
  SHC_PTR(pairs, "pairs");
  SHC_PTR(ws, "ws");
  const size_t need = shc_build_slot_pairs_workspace(n_rows, K);
  if (ws_bytes < need)
    return fail(SHC_ERR_CAPACITY, "workspace of %zu bytes is below the %zu needed", ws_bytes, need);
  return hip_status(shc::launch_slot_pairs(table, n_rows, K, pairs, pair_ptr, ws, stream),
                    "build_slot_pairs launch");
}

int shc_sparse_neighbor_conv_backward(const void* S, const int32_t* table, const int32_t* pairs,
                                      const int32_t* pair_ptr, const int32_t* table_t,
                                      const uint64_t* row_slots, const int32_t* slot_of,
                                      int32_t Kt, const void* W, const void* Y, const void* dY,
                                      int64_t n_rows, int32_t K, int32_t Cin, int32_t Cout,
                                      int32_t dtype, int32_t act, void* dS, float* dW, float* db,
                                      void* ws, size_t ws_bytes, hipStream_t stream) {
  g_last_error[0] = 0;
  if (K <= 0) return fail(SHC_ERR_INVALID_ARG, "K = %d must be positive", K);
  if (K > kMaxSlots) return fail(SHC_ERR_UNSUPPORTED, "K = %d exceeds %d slots", K, kMaxSlots);
  SHC_TRY(check_backward(S, W, Y, dY, n_rows, K, Cin, Cout, dtype, act, dS, dW, db, ws, ws_bytes,
                         shc_sparse_neighbor_conv_backward_workspace(n_rows, K, Cin, Cout, dtype)));
  if ((int64_t)K * n_rows > INT32_MAX)
    return fail(SHC_ERR_UNSUPPORTED, "K * n_rows exceeds 2^31 - 1");
  if ((pairs == nullptr) != (pair_ptr == nullptr))
    return fail(SHC_ERR_INVALID_ARG, "pairs and pair_ptr go together");
  SHC_OPT_PTR(pairs, "pairs");
  SHC_OPT_PTR(pair_ptr, "pair_ptr");
  if (n_rows > 0 && dW != nullptr) SHC_PTR(table, "table");
  if (n_rows > 0 && dS != nullptr) {
    if (Kt < 1 || Kt > SHC_MAX_VIRTUAL_SLOTS)
      return fail(SHC_ERR_INVALID_ARG, "Kt = %d outside [1, %d]", Kt, SHC_MAX_VIRTUAL_SLOTS);
    SHC_PTR(table_t, "table_t");
    SHC_PTR(row_slots, "row_slots");
    SHC_PTR(slot_of, "slot_of");
  }
  return hip_status(shc::launch_layer_backward(1, S, table, pairs, pair_ptr, table_t, row_slots,
                                               slot_of, W, Y, dY, n_rows, K, Cin, Cout,
                                               dtype == SHC_BF16, act, dS, dW, db, ws, stream),
                    "sparse_neighbor_conv_backward launch");
}

int shc_segment_maxpool(const void* S, const int32_t* row_ptr, int64_t n_rows, int32_t B,
                        int32_t C, int32_t dtype, float empty_value, void* P, hipStream_t stream) {
  g_last_error[0] = 0;
  if (B <= 0) return fail(SHC_ERR_INVALID_ARG, "B = %d must be positive", B);
  SHC_TRY(check_rows(n_rows));
  SHC_TRY(check_dtype(dtype));
  SHC_TRY(check_channels("C", C));
  SHC_PTR(row_ptr, "row_ptr");
  SHC_PTR(P, "P");
  if (n_rows > 0) SHC_PTR(S, "S");
  return hip_status(shc::launch_segment_max(S, row_ptr, n_rows, B, C, dtype == SHC_BF16,
                                            empty_value, P, stream),
                    "segment_maxpool launch");
}

// -- stream-ordering events ---------------------------------------------------

int shc_event_create(void** event) {
  g_last_error[0] = 0;
  if (event == nullptr) return fail(SHC_ERR_INVALID_ARG, "event is NULL");
  *event = nullptr;
  hipEvent_t ev = nullptr;
  SHC_TRY(hip_status(hipEventCreateWithFlags(&ev, hipEventDisableTiming | hipEventDisableSystemFence),
                     "event create"));
  *event = ev;
  return SHC_OK;
}

int shc_event_record(void* event, hipStream_t stream) {
  g_last_error[0] = 0;
  if (event == nullptr) return fail(SHC_ERR_INVALID_ARG, "event is NULL");
  return hip_status(hipEventRecord(static_cast<hipEvent_t>(event), stream), "event record");
}

int shc_stream_wait_event(hipStream_t stream, void* event) {
  g_last_error[0] = 0;
  if (event == nullptr) return fail(SHC_ERR_INVALID_ARG, "event is NULL");
  return hip_status(hipStreamWaitEvent(stream, static_cast<hipEvent_t>(event), 0),
                    "stream wait event");
}

int shc_event_synchronize(void* event) {
  g_last_error[0] = 0;
  if (event == nullptr) return fail(SHC_ERR_INVALID_ARG, "event is NULL");
  return hip_status(hipEventSynchronize(static_cast<hipEvent_t>(event)), "event synchronize");
}

int shc_event_destroy(void* event) {
  g_last_error[0] = 0;
  if (event == nullptr) return SHC_OK;
  return hip_status(hipEventDestroy(static_cast<hipEvent_t>(event)), "event destroy");
}

}  // extern "C"
