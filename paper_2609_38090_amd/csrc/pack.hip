// Device packer: fp32/bf16 expert weights -> packed experts (paper section
// IV-B).  Per expert-hidden row r:
//   alpha_r = max(|gate[r,:]|_inf, |up[r,:]|_inf, |down[:,r]|_inf)
//   sigma_r = bf16_rne(fl32(max(alpha_r, eps) / 127))
//   q       = clamp(rint_even(fl32(w / sigma_r)), -127, 127)
// The division is the IEEE correctly rounded fp32 one (this file is built
// without fast-math), so the bytes equal the host packer's.
#include "device_util.h"
#include "int4_format.h"
#include "mira_internal.h"

namespace mira {

template <typename WT>
__device__ __forceinline__ float ldw(const WT* p, size_t i);
template <>
__device__ __forceinline__ float ldw<float>(const float* p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ldw<uint16_t>(const uint16_t* p, size_t i) {
  return bf16_to_f32(p[i]);
}

// amax[e][r] = max over gate row r and up row r (one wave per row)
template <typename WT>
__global__ __launch_bounds__(256) void pack_rowmax_kernel(const WT* __restrict__ wg,
                                                          const WT* __restrict__ wu, int C, int R,
                                                          uint32_t* __restrict__ amax) {
  const int e = blockIdx.y;
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= R) return;
  const size_t base = ((size_t)e * R + r) * C;
  float m = 0.f;
  for (int c = lane; c < C; c += 64) m = fmaxf(m, fmaxf(fabsf(ldw(wg, base + c)), fabsf(ldw(wu, base + c))));
  m = wave_max(m);
  if (lane == 0) amax[(size_t)e * R + r] = __float_as_uint(m);
}

// amax[e][r] = max(amax[e][r], max over a chunk of c of |down[c][r]|)
template <typename WT>
__global__ __launch_bounds__(256) void pack_colmax_kernel(const WT* __restrict__ wd, int C, int R,
                                                          int c_chunk, uint32_t* __restrict__ amax) {
  const int e = blockIdx.z;
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= R) return;
  const int c0 = blockIdx.y * c_chunk, c1 = min(C, c0 + c_chunk);
  const WT* p = wd + (size_t)e * C * R + r;
  float m = 0.f;
  for (int c = c0; c < c1; ++c) m = fmaxf(m, fabsf(ldw(p, (size_t)c * R)));
  // non-negative floats order like their bit patterns
  atomicMax(&amax[(size_t)e * R + r], __float_as_uint(m));
}

__device__ __forceinline__ float scale_of(uint32_t amax_bits, float eps) {
  const float s32 = fmaxf(__uint_as_float(amax_bits), eps) / 127.0f;
  return bf16_to_f32(f32_to_bf16_rne(s32));
}

__device__ __forceinline__ int8_t quant(float w, float sigma) {
  float q = rintf(w / sigma);
  q = fminf(fmaxf(q, -127.f), 127.f);
  return (int8_t)(int)q;
}

// gate/up rows: blob[e] bytes [0, 2RC) in the tiled layout; one workgroup per (row, matrix)
template <typename WT>
__global__ __launch_bounds__(256) void pack_quant_rows_kernel(const WT* __restrict__ wg,
                                                              const WT* __restrict__ wu, int C,
                                                              int R, float eps,
                                                              const uint32_t* __restrict__ amax,
                                                              int8_t* __restrict__ packed,
                                                              uint64_t stride) {
  const int e = blockIdx.z, mat = blockIdx.y, r = blockIdx.x;
  const float sigma = scale_of(amax[(size_t)e * R + r], eps);
  const WT* src = (mat == 0 ? wg : wu) + ((size_t)e * R + r) * C;
  int8_t* dst = packed + (size_t)e * stride + (size_t)mat * R * C;
  for (int c = threadIdx.x; c < C; c += 256) dst[tiled_offset(r, c, C)] = quant(ldw(src, c), sigma);
}

// down [C][R]: column r uses sigma_r; also writes sigma and zero padding
template <typename WT>
__global__ __launch_bounds__(256) void pack_quant_down_kernel(const WT* __restrict__ wd, int C,
                                                              int R, float eps,
                                                              const uint32_t* __restrict__ amax,
                                                              int8_t* __restrict__ packed,
                                                              uint64_t stride) {
  const int e = blockIdx.z, c = blockIdx.y;
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= R) return;
  const float sigma = scale_of(amax[(size_t)e * R + r], eps);
  int8_t* blob = packed + (size_t)e * stride;
  blob[(size_t)2 * R * C + tiled_offset(c, r, R)] = quant(ldw(wd, ((size_t)e * C + c) * R + r), sigma);
  if (c == 0) {
    uint16_t* sig = (uint16_t*)(blob + (size_t)3 * R * C);
    sig[r] = f32_to_bf16_rne(fmaxf(__uint_as_float(amax[(size_t)e * R + r]), eps) / 127.0f);
  }
}

__global__ __launch_bounds__(256) void pack_pad_kernel(int8_t* __restrict__ packed, uint64_t stride,
                                                       uint64_t used) {
  const int e = blockIdx.y;
  for (uint64_t i = used + (uint64_t)blockIdx.x * 256 + threadIdx.x; i < stride;
       i += (uint64_t)gridDim.x * 256)
    packed[(size_t)e * stride + i] = 0;
}

// INT4 variant: one thread per (row, group of 64 columns) of one matrix of one
// expert; it owns the group's 32 nibble bytes (four 8-byte half-runs) and its
// scale.
template <typename WT>
__global__ __launch_bounds__(256) void pack_i4_kernel(const WT* __restrict__ wg,
                                                      const WT* __restrict__ wu,
                                                      const WT* __restrict__ wd, int C, int R,
                                                      float eps, uint8_t* __restrict__ packed,
                                                      uint64_t stride) {
  const int mat = blockIdx.y, e = blockIdx.z;
  const int rows = mat == 2 ? C : R, K = mat == 2 ? R : C;
  const int groups = K / 64;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (int64_t)rows * groups) return;
  const int r = (int)(idx / groups), blk = (int)(idx - (int64_t)r * groups);
  const WT* src = (mat == 0 ? wg : mat == 1 ? wu : wd) + (size_t)e * R * C + (size_t)r * K + blk * 64;
  float w[64];
  float alpha = 0.f;
#pragma unroll
  for (int c = 0; c < 64; ++c) {
    w[c] = ldw(src, c);
    alpha = fmaxf(alpha, fabsf(w[c]));
  }
  const uint16_t sb = i4_scale_bits(fmaxf(alpha, eps) / (float)kI4QMax);
  const float s = i4_scale_value(sb);
  uint8_t* blob = packed + (size_t)e * stride + (size_t)mat * i4_matrix_bytes(R, C);  // gate, up, down
#pragma unroll
  for (int gq = 0; gq < 4; ++gq) {
    uint64_t run = 0;
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const int c = 16 * gq + 8 * (b >> 2) + (b & 3);
      const int qh = (int)fminf(fmaxf(rintf(w[c] / s), -(float)kI4QMax), (float)kI4QMax);
      const int ql = (int)fminf(fmaxf(rintf(w[c + 4] / s), -(float)kI4QMax), (float)kI4QMax);
      run |= (uint64_t)(((qh & 0xF) << 4) | (ql & 0xF)) << (8 * b);
    }
    *(uint64_t*)(blob + i4_half_run_offset(r, blk, gq, K)) = run;
  }
  *(uint16_t*)(blob + i4_scale_offset(r, blk, rows, K)) = sb;
}

hipError_t launch_pack_i4(int C, int R, int n, int w_dtype, const void* wg, const void* wu,
                          const void* wd, float eps, void* packed, uint64_t stride,
                          hipStream_t st) {
  if (n == 0) return hipSuccess;
  prof_begin("pack", st);
  const int64_t items = (int64_t)R * (C / 64);  // rows x groups, the same for all three matrices
  const dim3 grid((unsigned)((items + 255) / 256), 3, n);
  if (w_dtype == MIRA_BF16)
    hipLaunchKernelGGL(pack_i4_kernel<uint16_t>, grid, dim3(256), 0, st, (const uint16_t*)wg,
                       (const uint16_t*)wu, (const uint16_t*)wd, C, R, eps, (uint8_t*)packed, stride);
  else
    hipLaunchKernelGGL(pack_i4_kernel<float>, grid, dim3(256), 0, st, (const float*)wg,
                       (const float*)wu, (const float*)wd, C, R, eps, (uint8_t*)packed, stride);
  const uint64_t used = 2 * i4_matrix_bytes(R, C) + i4_matrix_bytes(C, R);
  if (stride > used)
    hipLaunchKernelGGL(pack_pad_kernel, dim3(64, n), dim3(256), 0, st, (int8_t*)packed, stride, used);
  prof_end("pack", st);
  return hipGetLastError();
}

hipError_t launch_pack(int C, int R, int n, int w_dtype, const void* wg, const void* wu,
                       const void* wd, float eps, void* packed, uint64_t stride, hipStream_t st) {
  if (n == 0) return hipSuccess;
  // fp32 row maxima alpha_r live in a stream-ordered temporary allocation
  // (packing is offline; the forward path never allocates).
  uint32_t* amax = nullptr;
  hipError_t err = hipMallocAsync((void**)&amax, (size_t)n * R * 4, st);
  if (err != hipSuccess) return err;
  prof_begin("pack", st);
  const int c_chunk = 256;
  if (w_dtype == MIRA_BF16) {
    const uint16_t *g = (const uint16_t*)wg, *u = (const uint16_t*)wu, *d = (const uint16_t*)wd;
    hipLaunchKernelGGL(pack_rowmax_kernel<uint16_t>, dim3((R + 3) / 4, n), dim3(256), 0, st, g, u,
                       C, R, amax);
    hipLaunchKernelGGL(pack_colmax_kernel<uint16_t>, dim3((R + 255) / 256, (C + c_chunk - 1) / c_chunk, n),
                       dim3(256), 0, st, d, C, R, c_chunk, amax);
    hipLaunchKernelGGL(pack_quant_rows_kernel<uint16_t>, dim3(R, 2, n), dim3(256), 0, st, g, u, C,
                       R, eps, amax, (int8_t*)packed, stride);
    hipLaunchKernelGGL(pack_quant_down_kernel<uint16_t>, dim3((R + 255) / 256, C, n), dim3(256), 0,
                       st, d, C, R, eps, amax, (int8_t*)packed, stride);
  } else {
    const float *g = (const float*)wg, *u = (const float*)wu, *d = (const float*)wd;
    hipLaunchKernelGGL(pack_rowmax_kernel<float>, dim3((R + 3) / 4, n), dim3(256), 0, st, g, u, C,
                       R, amax);
    hipLaunchKernelGGL(pack_colmax_kernel<float>, dim3((R + 255) / 256, (C + c_chunk - 1) / c_chunk, n),
                       dim3(256), 0, st, d, C, R, c_chunk, amax);
    hipLaunchKernelGGL(pack_quant_rows_kernel<float>, dim3(R, 2, n), dim3(256), 0, st, g, u, C, R,
                       eps, amax, (int8_t*)packed, stride);
    hipLaunchKernelGGL(pack_quant_down_kernel<float>, dim3((R + 255) / 256, C, n), dim3(256), 0,
                       st, d, C, R, eps, amax, (int8_t*)packed, stride);
  }
  const uint64_t used = (uint64_t)3 * R * C + (uint64_t)2 * R;
  if (stride > used)
    hipLaunchKernelGGL(pack_pad_kernel, dim3(64, n), dim3(256), 0, st, (int8_t*)packed, stride, used);
  prof_end("pack", st);
  err = hipGetLastError();
  hipError_t e2 = hipFreeAsync(amax, st);
  return err != hipSuccess ? err : e2;
}

}  // namespace mira
