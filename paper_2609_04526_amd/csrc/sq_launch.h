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
                const uint8_t* codes, float* dS, hipStream_t s);

// One plane of a merge launch.
struct MergePlane {
  uint8_t* scales;
  const float* delta;
  const uint8_t* src;
  int64_t n;
  int64_t chunk_begin;   // first global chunk index of this plane
  float ws2;
  int32_t fmt;
  int32_t mode;
};
constexpr int kMergePlanesPerLaunch = 40;
constexpr int kMergeChunk = 4096;     // scale bytes per workgroup
struct MergeBatch {
  MergePlane p[kMergePlanesPerLaunch];
  int32_t count;
};
int merge_launch(const MergeBatch& b, int64_t total_chunks, hipStream_t s);

int rtn_launch(int fmt, int O, int I, const void* W, float ws2_in, int tie,
               uint8_t* codes, uint8_t* scales, float* ws2_out, hipStream_t s);

}  // namespace sq
