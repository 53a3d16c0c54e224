// Internal host-side interface between the C-ABI layer (api.hip) and the
// kernel translation units.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace elas {

// Row pitches of the compressed 2:4 layout: rows are padded to a multiple of
// 64 features (32 kept values, 8 metadata bytes per 64 features).
inline int64_t vals_ld(int64_t n) { return 32 * ((n + 63) / 64); }
inline int64_t meta_ld(int64_t n) { return 8 * ((n + 63) / 64); }
inline int64_t pad64(int64_t n) { return 64 * ((n + 63) / 64); }
inline int64_t pad256(int64_t n) { return 256 * ((n + 255) / 256); }

// timing.hip: brackets one launch with events when timing is enabled, and
// synchronises after it in the ELAS_DEBUG_SYNC mode (the first failure of
// the calling thread is kept with its kernel tag until the next reset)
bool timing_enabled();
void debug_sync_reset();
hipError_t debug_sync_error(const char** tag);
class TimedLaunch {
 public:
  TimedLaunch(const char* tag, hipStream_t stream);
  ~TimedLaunch();
  TimedLaunch(const TimedLaunch&) = delete;
  TimedLaunch& operator=(const TimedLaunch&) = delete;

 private:
  const char* tag_;
  hipStream_t stream_;
  hipEvent_t start_ = nullptr, stop_ = nullptr;
};

// sparsify.hip
hipError_t launch_sparsify24(const uint16_t* h, int64_t M, int64_t N, bool raw,
                             uint16_t* vals, uint8_t* meta, hipStream_t stream);

// Arguments of one forward or backward call (sizes already validated).
struct FfnArgs {
  int64_t T, d, F, r;
  const uint16_t *x, *U_up, *V_up, *U_down, *V_down;
  // forward outputs / backward inputs
  uint16_t* y;
  const uint16_t* P_in;
  uint16_t* P;
  uint16_t* s_vals;
  uint8_t* s_meta;
  uint16_t* Z;
  // backward
  const uint16_t* dy;
  uint16_t* dx;
  float *dU_up, *dV_up, *dU_down, *dV_down;
  void* ws;
  bool dense;   // activations dense [T x d_ff] (no 2:4 selection)
  bool ste;     // backward: straight-through estimator through the selection
  bool ab;      // forward: factors given as U_up^T, V_up^T, U_down^T, V_down^T
  int fused;    // sparse forward: 1 one fused launch, else (0 default, 2 requested) four kernels
};

// fused.hip: the one-launch sparse forward for compact factor shapes
bool fused_fwd_supported(int64_t d, int64_t r);
hipError_t run_fused_fwd(const uint16_t* x, const uint16_t* U_upT, const uint16_t* V_upT, const uint16_t* U_downT,
                         const uint16_t* V_downT, int64_t T, int64_t d, int64_t F, int64_t r, int64_t F_rows,
                         int64_t ld_ud, uint16_t* y, uint16_t* P, uint16_t* s_vals, uint8_t* s_meta, uint16_t* Z,
                         hipStream_t stream);

// ffn.hip
size_t spmm_workspace_bytes(int64_t K, int64_t N, int b_layout);
size_t fwd_workspace_bytes(int64_t T, int64_t d, int64_t F, int64_t r, bool dense, bool ab);
size_t bwd_workspace_bytes(int64_t T, int64_t d, int64_t F, int64_t r, bool dense, bool ste);
hipError_t run_spmm24(const uint16_t* a_vals, const uint8_t* a_meta, int64_t M, int64_t K,
                      const uint16_t* b, int64_t N, bool b_is_nk, uint16_t* c, void* ws,
                      hipStream_t stream);
hipError_t run_fwd(const FfnArgs& a, hipStream_t stream);
hipError_t run_bwd(const FfnArgs& a, hipStream_t stream);
hipError_t run_fullrank_fwd(const uint16_t* x, const uint16_t* W_up, const uint16_t* W_down, int64_t T,
                            int64_t d, int64_t F, uint16_t* y, uint16_t* S, hipStream_t stream);

}  // namespace elas
