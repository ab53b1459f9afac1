// Online Hadamard rotation of rows, nq_rotate (Sec. 5 of the NestQuant paper): a workgroup
// holds R rows in LDS as fp32 (R n <= 2048 elements, or one row, with 256 threads; rows of
// more than 12288 entries with 1024 threads, whose extra waves keep more of the row's loads
// and stores in flight: at 56 to 128 KiB of LDS per row only one or two rows fit a CU),
// rotates them (nq_rotate.hpp) and writes y = (rotated entries) * fl32(1 / sqrt(n)).
#include <algorithm>
#include <cmath>

#include "nq_device.hpp"
#include "nq_kernels.hpp"
#include "nq_rotate.hpp"

namespace nq {

// Rows at least this long get a workgroup of 1024 threads.
constexpr int kRotateWideCols = 12288;

// With 1024 threads, at most 64 VGPRs, so that two rows (two workgroups) fit a CU while
// their LDS does (n <= 14336): one row's loads and stores then overlap the other's transform.
template <typename T, int NT>
__global__ __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(NT == 1024 ? 8 : 1)))
void rotate_kernel(const T* __restrict__ x, int64_t rows, int n, int64_t ld_x, int p, int lp,
                   int rpw, float s, float* __restrict__ y, int64_t ld_y) {
  extern __shared__ float buf[];
  const int tid = threadIdx.x;
  const int64_t row0 = (int64_t)blockIdx.x * rpw;
  const int rr = (int)std::min<int64_t>(rpw, rows - row0);   // rows in this workgroup
  const int total = rr * n;                                  // elements held
  const int half = rotate_rows_lds<T, NT, true>(x + row0 * ld_x, ld_x, rr, n, p, lp, buf);
  if (half > 0) {
    // the last stage, h = half (a power of two >= 8), fused with the output: entries e and
    // e + half of each group of 8 become (a + b, a - b), then times s
    for (int g = 8 * tid; g < total / 2; g += 8 * NT) {
      const int e = ((g & -half) << 1) | (g & (half - 1));
      const int r = rr == 1 ? 0 : e / n, c = e - r * n;
      const int pa = lds_pos(e), pb = lds_pos(e + half);
      float lo[8], hi[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const float a = buf[pa ^ i], b = buf[pb ^ i];
        lo[i] = (a + b) * s;
        hi[i] = (a - b) * s;
      }
      f32x4* o = reinterpret_cast<f32x4*>(y + (row0 + r) * ld_y + c);
      __builtin_nontemporal_store((f32x4){lo[0], lo[1], lo[2], lo[3]}, o);
      __builtin_nontemporal_store((f32x4){lo[4], lo[5], lo[6], lo[7]}, o + 1);
      o = reinterpret_cast<f32x4*>(y + (row0 + r) * ld_y + c + half);
      __builtin_nontemporal_store((f32x4){hi[0], hi[1], hi[2], hi[3]}, o);
      __builtin_nontemporal_store((f32x4){hi[4], hi[5], hi[6], hi[7]}, o + 1);
    }
    return;
  }
  auto out = [&](int e, int r, int c) {
    const int pe = lds_pos(e);
    f32x4 lo = {buf[pe] * s, buf[pe ^ 1] * s, buf[pe ^ 2] * s, buf[pe ^ 3] * s};
    f32x4 hi = {buf[pe ^ 4] * s, buf[pe ^ 5] * s, buf[pe ^ 6] * s, buf[pe ^ 7] * s};
    f32x4* o = reinterpret_cast<f32x4*>(y + (row0 + r) * ld_y + c);
    __builtin_nontemporal_store(lo, o);
    __builtin_nontemporal_store(hi, o + 1);
  };
  if (rr == 1) {
    for (int e = 8 * tid; e < n; e += 8 * NT) out(e, 0, e);
  } else {
    for (int e = 8 * tid; e < total; e += 8 * NT) {
      const int r = e / n;
      out(e, r, e - r * n);
    }
  }
}

template <typename T>
static hipError_t launch_t(const void* x, int64_t rows, int n, int64_t ld_x, float* y,
                           int64_t ld_y, hipStream_t st) {
  int p = 0;
  rotation_split(n, p);
  int lp = 0;
  while ((1 << lp) < p) ++lp;
  const int rpw = n >= 2048 ? 1 : 2048 / n;
  const size_t lds = (size_t)rpw * n * sizeof(float);
  const float s = (float)(1.0 / std::sqrt((double)n));
  const int64_t grid = (rows + rpw - 1) / rpw;
  if (n >= kRotateWideCols) {
    hipLaunchKernelGGL((rotate_kernel<T, 1024>), dim3((unsigned)grid), dim3(1024), lds, st,
                       (const T*)x, rows, n, ld_x, p, lp, rpw, s, y, ld_y);
  } else {
    hipLaunchKernelGGL((rotate_kernel<T, 256>), dim3((unsigned)grid), dim3(256), lds, st,
                       (const T*)x, rows, n, ld_x, p, lp, rpw, s, y, ld_y);
  }
  return hipGetLastError();
}

hipError_t rotate_set_attributes() {
  const void* k[6] = {(const void*)rotate_kernel<float, 256>, (const void*)rotate_kernel<_Float16, 256>,
                      (const void*)rotate_kernel<uint16_t, 256>, (const void*)rotate_kernel<float, 1024>,
                      (const void*)rotate_kernel<_Float16, 1024>, (const void*)rotate_kernel<uint16_t, 1024>};
  for (int i = 0; i < 6; ++i) {
    const hipError_t e = hipFuncSetAttribute(k[i], hipFuncAttributeMaxDynamicSharedMemorySize,
                                             kRotateMaxCols * (int)sizeof(float));
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

hipError_t launch_rotate(const void* x, int dtype, int64_t rows, int n, int64_t ld_x, float* y,
                         int64_t ld_y, hipStream_t st) {
  switch (dtype) {
    case 0: return launch_t<float>(x, rows, n, ld_x, y, ld_y, st);
    case 1: return launch_t<_Float16>(x, rows, n, ld_x, y, ld_y, st);
    default: return launch_t<uint16_t>(x, rows, n, ld_x, y, ld_y, st);
  }
}

}  // namespace nq
