// C-ABI layer of libelas: argument validation, workspace carving and launch
// orchestration on the caller's stream.  Every check runs on the host before
// anything is enqueued, so an error leaves outputs untouched.
#include <stdarg.h>
#include <stdio.h>

#include <mutex>
#include <string>

#include "../../include/elas.h"
#include "internal.h"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// NULL / alignment check of one device pointer.
int check_ptr(const void* p, const char* name) {
  if (p == nullptr) return fail(ELAS_ERR_NULL, "%s is NULL", name);
  if (!aligned16(p)) return fail(ELAS_ERR_ALIGN, "%s is not 16-byte aligned", name);
  return ELAS_OK;
}

#define ELAS_CHECK(expr)            \
  do {                              \
    int rc_ = (expr);               \
    if (rc_ != ELAS_OK) return rc_; \
  } while (0)

// Status of a launch sequence: its own error, else (ELAS_DEBUG_SYNC) the
// first failure seen when synchronising after one of its kernels.
int device_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(ELAS_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
  const char* tag = nullptr;
  const hipError_t d = elas::debug_sync_error(&tag);
  if (d != hipSuccess)
    return fail(ELAS_ERR_DEVICE, "%s: kernel %s failed (ELAS_DEBUG_SYNC): %s", what, tag ? tag : "?",
                hipGetErrorString(d));
  return ELAS_OK;
}

// Sizes are bounded so every element offset fits comfortably in int64 and in
// the 32-bit grid dimensions used by the launchers.
constexpr int64_t kMaxDim = int64_t(1) << 31;

int check_ffn_dims(int64_t T, int64_t d, int64_t d_ff, int64_t r) {
  if (T < 0 || T > kMaxDim) return fail(ELAS_ERR_SHAPE, "T=%lld out of range", (long long)T);
  if (d <= 0 || d % 8) return fail(ELAS_ERR_SHAPE, "d=%lld must be a positive multiple of 8", (long long)d);
  if (d_ff <= 0 || d_ff % 8)
    return fail(ELAS_ERR_SHAPE, "d_ff=%lld must be a positive multiple of 8", (long long)d_ff);
  if (r <= 0 || r % 8) return fail(ELAS_ERR_SHAPE, "r=%lld must be a positive multiple of 8", (long long)r);
  if (d > 65536 || d_ff > 65536 || r > 65536)
    return fail(ELAS_ERR_SHAPE, "d, d_ff and r must be at most 65536");
  return ELAS_OK;
}

// Host-side conversion of the tiled compressed layout (the FFN's saved S) to
// the canonical one: entry j of row i sits at tiled element
// (i / 256) * 256 * ld + (j / BW) * R * BW + (i % 256) * BW + j % BW,
// R = the rows of i's block of 256.
template <class E, int BW>
int tiled_to_canonical(const E* tiled, int64_t M, int64_t ld, int64_t n_out, E* out, const char* what) {
  g_last_error.clear();
  if (M < 0 || M > kMaxDim) return fail(ELAS_ERR_SHAPE, "M=%lld out of range", (long long)M);
  if (M == 0) return ELAS_OK;
  if (tiled == nullptr || out == nullptr) return fail(ELAS_ERR_NULL, "%s: NULL buffer", what);
  for (int64_t i = 0; i < M; ++i) {
    const int64_t b = i / 256, R = M - b * 256 < 256 ? M - b * 256 : 256;
    const E* blk = tiled + b * 256 * ld;
    for (int64_t j = 0; j < n_out; ++j) out[i * n_out + j] = blk[(j / BW) * R * BW + (i % 256) * BW + j % BW];
  }
  return ELAS_OK;
}
// Checks of the forward's arguments shared by its two entry points; fills
// the launch arguments (without workspace).  noop: T == 0, nothing to do.
int prepare_fwd(const uint16_t* x, const uint16_t* U_up, const uint16_t* V_up, const uint16_t* U_down,
                const uint16_t* V_down, int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags, uint16_t* y,
                uint16_t* P, uint16_t* s_vals, uint8_t* s_meta, uint16_t* Z, elas::FfnArgs& a, bool& noop) {
  if (flags & ~(ELAS_MODE_DENSE | ELAS_FACTORS_AB | ELAS_FWD_FUSED | ELAS_FWD_UNFUSED))
    return fail(ELAS_ERR_FLAGS,
                "forward flags: only ELAS_MODE_DENSE, ELAS_FACTORS_AB, ELAS_FWD_FUSED and ELAS_FWD_UNFUSED are allowed");
  const bool dense = (flags & ELAS_MODE_DENSE) != 0, ab = (flags & ELAS_FACTORS_AB) != 0;
  const bool fused = (flags & ELAS_FWD_FUSED) != 0, unfused = (flags & ELAS_FWD_UNFUSED) != 0;
  if (fused && unfused) return fail(ELAS_ERR_FLAGS, "ELAS_FWD_FUSED and ELAS_FWD_UNFUSED exclude each other");
  if (fused && dense) return fail(ELAS_ERR_FLAGS, "ELAS_FWD_FUSED applies to the sparse forward only");
  ELAS_CHECK(check_ffn_dims(T, d, d_ff, r));
  if (fused && !elas::fused_fwd_supported(d, r))
    return fail(ELAS_ERR_SHAPE, "ELAS_FWD_FUSED needs d a multiple of 64 up to 1024 and r = 128 or 256 (d=%lld r=%lld)",
                (long long)d, (long long)r);
  noop = T == 0;
  if (noop) return ELAS_OK;
  ELAS_CHECK(check_ptr(x, "x"));
  ELAS_CHECK(check_ptr(U_up, "U_up"));
  ELAS_CHECK(check_ptr(V_up, "V_up"));
  ELAS_CHECK(check_ptr(U_down, "U_down"));
  ELAS_CHECK(check_ptr(V_down, "V_down"));
  ELAS_CHECK(check_ptr(y, "y"));
  ELAS_CHECK(check_ptr(P, "P"));
  ELAS_CHECK(check_ptr(s_vals, "s_vals"));
  if (!dense) ELAS_CHECK(check_ptr(s_meta, "s_meta"));
  ELAS_CHECK(check_ptr(Z, "Z"));
  a.T = T; a.d = d; a.F = d_ff; a.r = r;
  a.x = x; a.U_up = U_up; a.V_up = V_up; a.U_down = U_down; a.V_down = V_down;
  a.y = y; a.P = P; a.P_in = P; a.s_vals = s_vals; a.s_meta = s_meta; a.Z = Z;
  a.dense = dense;
  a.ab = ab;
  a.fused = fused ? 1 : unfused ? 2 : 0;
  return ELAS_OK;
}

// Workspace of elas_lowrank_ffn_fwd_noalloc: one static array per device,
// held until the process ends.  Its device address is looked up once per
// device (with that device current) and kept; the array's name is only a
// host-side stand-in and is never passed to a kernel.
constexpr size_t kScratchBytes = ELAS_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

int scratch_address(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(ELAS_ERR_DEVICE, "hipGetDevice: %s", hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(ELAS_ERR_DEVICE, "device %d beyond the supported %d", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(ELAS_ERR_DEVICE, "hipGetSymbolAddress(scratch) on device %d: %s", dev, hipGetErrorString(e));
    g_scratch[dev] = p;
  }
  *out = g_scratch[dev];
  return ELAS_OK;
}

}  // namespace

extern "C" {

const char* elas_status_string(int status) {
  switch (status) {
    case ELAS_OK: return "ELAS_OK";
    case ELAS_ERR_NULL: return "ELAS_ERR_NULL";
    case ELAS_ERR_SHAPE: return "ELAS_ERR_SHAPE";
    case ELAS_ERR_ALIGN: return "ELAS_ERR_ALIGN";
    case ELAS_ERR_WORKSPACE: return "ELAS_ERR_WORKSPACE";
    case ELAS_ERR_FLAGS: return "ELAS_ERR_FLAGS";
    case ELAS_ERR_DEVICE: return "ELAS_ERR_DEVICE";
    default: return "ELAS_ERR_UNKNOWN";
  }
}

const char* elas_last_error(void) { return g_last_error.c_str(); }

int64_t elas_vals_ld(int64_t N) { return N > 0 ? elas::vals_ld(N) : 0; }
int64_t elas_meta_ld(int64_t N) { return N > 0 ? elas::meta_ld(N) : 0; }

int elas_sparsify_24(const uint16_t* h, int64_t M, int64_t N, uint32_t flags, uint16_t* vals,
                     uint8_t* meta, void* stream) {
  g_last_error.clear();
  elas::debug_sync_reset();
  if (flags & ~ELAS_SPARSIFY_RAW) return fail(ELAS_ERR_FLAGS, "unknown flags 0x%x", flags);
  if (M < 0 || M > kMaxDim) return fail(ELAS_ERR_SHAPE, "M=%lld out of range", (long long)M);
  if (N <= 0 || N % 8 || N > kMaxDim)
    return fail(ELAS_ERR_SHAPE, "N=%lld must be a positive multiple of 8", (long long)N);
  if (M * (elas::vals_ld(N) / 8) >= (int64_t(1) << 40))
    return fail(ELAS_ERR_SHAPE, "M*N too large");
  if (M == 0) return ELAS_OK;
  ELAS_CHECK(check_ptr(h, "h"));
  ELAS_CHECK(check_ptr(vals, "vals"));
  ELAS_CHECK(check_ptr(meta, "meta"));
  return device_status(
      elas::launch_sparsify24(h, M, N, (flags & ELAS_SPARSIFY_RAW) != 0, vals, meta, (hipStream_t)stream),
      "sparsify launch");
}

size_t elas_spmm_24_workspace_bytes(int64_t M, int64_t K, int64_t N, int b_layout) {
  (void)M;
  if (K <= 0 || N <= 0) return 0;
  return elas::spmm_workspace_bytes(K, N, b_layout);
}

int elas_spmm_24(const uint16_t* a_vals, const uint8_t* a_meta, int64_t M, int64_t K, const uint16_t* b,
                 int64_t N, int b_layout, uint16_t* c, void* workspace, size_t workspace_bytes,
                 void* stream) {
  g_last_error.clear();
  elas::debug_sync_reset();
  if (b_layout != ELAS_B_KN && b_layout != ELAS_B_NK)
    return fail(ELAS_ERR_FLAGS, "b_layout must be ELAS_B_KN or ELAS_B_NK");
  if (M < 0 || M > kMaxDim) return fail(ELAS_ERR_SHAPE, "M=%lld out of range", (long long)M);
  if (K <= 0 || K % 8 || K > 65536)
    return fail(ELAS_ERR_SHAPE, "K=%lld must be a positive multiple of 8, at most 65536", (long long)K);
  if (N <= 0 || N % 8 || N > 65536)
    return fail(ELAS_ERR_SHAPE, "N=%lld must be a positive multiple of 8, at most 65536", (long long)N);
  if (M == 0) return ELAS_OK;
  ELAS_CHECK(check_ptr(a_vals, "a_vals"));
  ELAS_CHECK(check_ptr(a_meta, "a_meta"));
  ELAS_CHECK(check_ptr(b, "b"));
  ELAS_CHECK(check_ptr(c, "c"));
  const size_t need = elas::spmm_workspace_bytes(K, N, b_layout);
  if (workspace_bytes < need)
    return fail(ELAS_ERR_WORKSPACE, "workspace %zu bytes, %zu needed", workspace_bytes, need);
  if (need) ELAS_CHECK(check_ptr(workspace, "workspace"));
  return device_status(elas::run_spmm24(a_vals, a_meta, M, K, b, N, b_layout == ELAS_B_NK, c, workspace,
                                        (hipStream_t)stream),
                       "spmm launch");
}

size_t elas_lowrank_ffn_fwd_workspace_bytes(int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags) {
  if (T < 0 || d <= 0 || d_ff <= 0 || r <= 0) return 0;
  return elas::fwd_workspace_bytes(T, d, d_ff, r, (flags & ELAS_MODE_DENSE) != 0, (flags & ELAS_FACTORS_AB) != 0);
}

int elas_lowrank_ffn_fwd(const uint16_t* x, const uint16_t* U_up, const uint16_t* V_up, const uint16_t* U_down,
                         const uint16_t* V_down, int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags,
                         uint16_t* y, uint16_t* P, uint16_t* s_vals, uint8_t* s_meta, uint16_t* Z,
                         void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  elas::debug_sync_reset();
  elas::FfnArgs a{};
  bool noop = false;
  ELAS_CHECK(prepare_fwd(x, U_up, V_up, U_down, V_down, T, d, d_ff, r, flags, y, P, s_vals, s_meta, Z, a, noop));
  if (noop) return ELAS_OK;
  const size_t need = elas::fwd_workspace_bytes(T, d, d_ff, r, a.dense, a.ab);
  if (workspace_bytes < need)
    return fail(ELAS_ERR_WORKSPACE, "workspace %zu bytes, %zu needed", workspace_bytes, need);
  if (need) ELAS_CHECK(check_ptr(workspace, "workspace"));
  a.ws = workspace;
  return device_status(elas::run_fwd(a, (hipStream_t)stream), "forward launch");
}

size_t elas_noalloc_scratch_bytes(void) { return kScratchBytes; }

int elas_lowrank_ffn_fwd_noalloc(const uint16_t* x, const uint16_t* U_up, const uint16_t* V_up,
                                 const uint16_t* U_down, const uint16_t* V_down, int64_t T, int64_t d, int64_t d_ff,
                                 int64_t r, uint32_t flags, uint16_t* y, uint16_t* P, uint16_t* s_vals,
                                 uint8_t* s_meta, uint16_t* Z, void* stream) {
  g_last_error.clear();
  elas::debug_sync_reset();
  elas::FfnArgs a{};
  bool noop = false;
  ELAS_CHECK(prepare_fwd(x, U_up, V_up, U_down, V_down, T, d, d_ff, r, flags, y, P, s_vals, s_meta, Z, a, noop));
  if (noop) return ELAS_OK;
  const size_t need = elas::fwd_workspace_bytes(T, d, d_ff, r, a.dense, a.ab);
  if (need > kScratchBytes)
    return fail(ELAS_ERR_WORKSPACE, "this forward needs %zu bytes of workspace; the static scratch holds %zu",
                need, kScratchBytes);
  void* ws = nullptr;
  if (need) ELAS_CHECK(scratch_address(&ws));
  a.ws = ws;
  return device_status(elas::run_fwd(a, (hipStream_t)stream), "forward launch (static scratch)");
}

size_t elas_lowrank_ffn_bwd_workspace_bytes(int64_t T, int64_t d, int64_t d_ff, int64_t r, uint32_t flags) {
  if (T < 0 || d <= 0 || d_ff <= 0 || r <= 0) return 0;
  return elas::bwd_workspace_bytes(T, d, d_ff, r, (flags & ELAS_MODE_DENSE) != 0, (flags & ELAS_BWD_STE) != 0);
}

int elas_lowrank_ffn_bwd(const uint16_t* dy, const uint16_t* x, const uint16_t* U_up, const uint16_t* V_up,
                         const uint16_t* U_down, const uint16_t* V_down, int64_t T, int64_t d, int64_t d_ff,
                         int64_t r, uint32_t flags, const uint16_t* P, const uint16_t* s_vals,
                         const uint8_t* s_meta, const uint16_t* Z, uint16_t* dx, float* dU_up, float* dV_up,
                         float* dU_down, float* dV_down, void* workspace, size_t workspace_bytes, void* stream) {
  g_last_error.clear();
  elas::debug_sync_reset();
  if (flags & ~(ELAS_MODE_DENSE | ELAS_BWD_STE))
    return fail(ELAS_ERR_FLAGS, "backward flags: only ELAS_MODE_DENSE or ELAS_BWD_STE are allowed");
  const bool dense = (flags & ELAS_MODE_DENSE) != 0, ste = (flags & ELAS_BWD_STE) != 0;
  if (dense && ste) return fail(ELAS_ERR_FLAGS, "ELAS_BWD_STE applies to the sparse forward only");
  ELAS_CHECK(check_ffn_dims(T, d, d_ff, r));
  if (T > 0) {   // with no tokens only the weight gradients (zeros) are written
    ELAS_CHECK(check_ptr(dy, "dy"));
    ELAS_CHECK(check_ptr(x, "x"));
    ELAS_CHECK(check_ptr(U_up, "U_up"));
    ELAS_CHECK(check_ptr(V_up, "V_up"));
    ELAS_CHECK(check_ptr(U_down, "U_down"));
    ELAS_CHECK(check_ptr(V_down, "V_down"));
    ELAS_CHECK(check_ptr(P, "P"));
    ELAS_CHECK(check_ptr(s_vals, "s_vals"));
    if (!dense) ELAS_CHECK(check_ptr(s_meta, "s_meta"));
    ELAS_CHECK(check_ptr(Z, "Z"));
    ELAS_CHECK(check_ptr(dx, "dx"));
  }
  ELAS_CHECK(check_ptr(dU_up, "dU_up"));
  ELAS_CHECK(check_ptr(dV_up, "dV_up"));
  ELAS_CHECK(check_ptr(dU_down, "dU_down"));
  ELAS_CHECK(check_ptr(dV_down, "dV_down"));
  const size_t need = elas::bwd_workspace_bytes(T, d, d_ff, r, dense, ste);
  if (workspace_bytes < need)
    return fail(ELAS_ERR_WORKSPACE, "workspace %zu bytes, %zu needed", workspace_bytes, need);
  if (need) ELAS_CHECK(check_ptr(workspace, "workspace"));
  elas::FfnArgs a{};
  a.T = T; a.d = d; a.F = d_ff; a.r = r;
  a.x = x; a.U_up = U_up; a.V_up = V_up; a.U_down = U_down; a.V_down = V_down;
  a.P = nullptr; a.P_in = P; a.s_vals = const_cast<uint16_t*>(s_vals);
  a.s_meta = const_cast<uint8_t*>(s_meta); a.Z = const_cast<uint16_t*>(Z);
  a.dy = dy; a.dx = dx; a.dU_up = dU_up; a.dV_up = dV_up; a.dU_down = dU_down; a.dV_down = dV_down;
  a.ws = workspace;
  a.dense = dense;
  a.ste = ste;
  return device_status(elas::run_bwd(a, (hipStream_t)stream), "backward launch");
}

int elas_fullrank_ffn_fwd(const uint16_t* x, const uint16_t* W_up, const uint16_t* W_down, int64_t T, int64_t d,
                          int64_t d_ff, uint16_t* y, uint16_t* S, void* stream) {
  g_last_error.clear();
  elas::debug_sync_reset();
  ELAS_CHECK(check_ffn_dims(T, d, d_ff, 8));
  if (T == 0) return ELAS_OK;
  ELAS_CHECK(check_ptr(x, "x"));
  ELAS_CHECK(check_ptr(W_up, "W_up"));
  ELAS_CHECK(check_ptr(W_down, "W_down"));
  ELAS_CHECK(check_ptr(y, "y"));
  ELAS_CHECK(check_ptr(S, "S"));
  return device_status(elas::run_fullrank_fwd(x, W_up, W_down, T, d, d_ff, y, S, (hipStream_t)stream),
                       "full-rank forward launch");
}


int elas_meta_to_canonical(const uint8_t* meta_tiled, int64_t M, int64_t N, uint8_t* meta_canonical) {
  if (N <= 0 || N % 8 || N > 65536) {
    g_last_error.clear();
    return fail(ELAS_ERR_SHAPE, "N=%lld must be a positive multiple of 8, at most 65536", (long long)N);
  }
  return tiled_to_canonical<uint8_t, 8>(meta_tiled, M, elas::meta_ld(N), N / 8, meta_canonical, "meta");
}

int elas_vals_to_canonical(const uint16_t* vals_tiled, int64_t M, int64_t N, uint16_t* vals_canonical) {
  if (N <= 0 || N % 8 || N > 65536) {
    g_last_error.clear();
    return fail(ELAS_ERR_SHAPE, "N=%lld must be a positive multiple of 8, at most 65536", (long long)N);
  }
  return tiled_to_canonical<uint16_t, 32>(vals_tiled, M, elas::vals_ld(N), N / 2, vals_canonical, "vals");
}

}  // extern "C"
