// Internal launchers behind the C ABI (all arguments already validated).
// Each returns 0 on success and -1 when the HIP runtime reports an error.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sq {

int gemm_fwd(int fmt, int T, int O, int I, const void* X, const uint8_t* codes,
             const uint8_t* scales, float ws2, void* Y, int y_bf16, hipStream_t s);
int gemm_dx(int fmt, int T, int O, int I, const void* dY, const uint8_t* codes,
            const uint8_t* scales, float ws2, void* dX, int dx_bf16, hipStream_t s);
int gemm_dscale(int fmt, int T, int O, int I, const void* X, const void* dY,
                const uint8_t* codes, float* dS, void* workspace, hipStream_t s);
// Workspace bytes gemm_dscale needs (partial dS planes of a split token sum).
size_t gemm_dscale_workspace(int fmt, int T, int O, int I);

// Planes of one merge launch, as arrays (kernel arguments are limited to
// 4 KiB; this layout fits 112 planes).  Plane p covers workgroups
// [chunk_begin[p], chunk_begin[p+1]).
constexpr int kMergePlanesPerLaunch = 112;
constexpr int kMergeUnit = 8192;      // workgroup chunks are multiples of this many scale bytes
struct MergeBatch {
  uint8_t* scales[kMergePlanesPerLaunch];
  const void* aux[kMergePlanesPerLaunch];     // fp32 delta (delta mode) or source bytes (copy mode)
  int64_t n[kMergePlanesPerLaunch];
  int32_t chunk_begin[kMergePlanesPerLaunch];
  float ws2[kMergePlanesPerLaunch];
  uint8_t fmt[kMergePlanesPerLaunch];
  uint8_t mode[kMergePlanesPerLaunch];
  int32_t count;
  int32_t chunk;                      // scale bytes per workgroup (a multiple of kMergeUnit)
};
static_assert(sizeof(MergeBatch) <= 4096, "kernel argument budget");
int merge_launch(const MergeBatch& b, int64_t total_chunks, hipStream_t s);
// Workgroup chunk for a launch over `total` scale bytes: enough workgroups to
// fill the chip, each large enough to amortise its set-up.
int64_t merge_chunk_for(int64_t total);

int rtn_launch(int fmt, int O, int I, const void* W, float ws2_in, int tie,
               uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s);

// QAST low-rank scale step: on-grid scale bytes (+ clamp mask) and the factor
// gradients; qast_grads_workspace bytes of partial dA planes.
int qast_scales_launch(int fmt, int O, int G, int r, const uint8_t* base, const void* B, const void* A,
                       float alpha_over_r, float ws2, uint8_t* out, uint8_t* mask, hipStream_t s);
size_t qast_grads_workspace(int O, int G, int r);
int qast_grads_launch(int O, int G, int r, const float* dS, const uint8_t* mask, const void* B, const void* A,
                      float alpha_over_r, float* dB, float* dA, void* workspace, hipStream_t s);

}  // namespace sq
