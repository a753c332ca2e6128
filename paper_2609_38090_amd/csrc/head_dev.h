// Row dot products of the predictor heads (section IV-E): one wave computes
// w . h_j for a bf16 weight row w of length C and up to NG pooled fp32 rows
// h_j.  The row is read with 16-byte loads, eight per lane issued before any
// arithmetic (4096 columns per pass), so a wave keeps 8 KB of weights in
// flight instead of waiting on one load at a time.
#pragma once

#include "device_util.h"

namespace mira {

constexpr int kHeadLoads = 8;                   // 16-byte loads per lane per pass
constexpr int kHeadPass = kHeadLoads * 64 * 8;  // columns per pass

// acc[j] += (this lane's share of) sum_c w[c] * h[j*C + c] for j < ng.
// C is a multiple of 8; w and h 16-byte aligned, h rows C floats apart.
template <int NG>
__device__ __forceinline__ void head_row_dot(const uint16_t* __restrict__ w,
                                             const float* __restrict__ h, int C, int ng, int lane,
                                             float (&acc)[NG]) {
  for (int c0 = 0; c0 < C; c0 += kHeadPass) {
    v4i q[kHeadLoads];
#pragma unroll
    for (int t = 0; t < kHeadLoads; ++t) {
      const int c = c0 + (t * 64 + lane) * 8;
      q[t] = c < C ? ld16(w + c) : zero16();
    }
#pragma unroll
    for (int j = 0; j < NG; ++j) {
      if (j < ng) {
        // this group's pooled values for the lane's columns, all loads issued
        // before the first product (zeros past the end of the row)
        v4f hv[2 * kHeadLoads];
#pragma unroll
        for (int t = 0; t < kHeadLoads; ++t) {
          const int c = c0 + (t * 64 + lane) * 8;
          const float* hp = h + (size_t)j * C + c;
          hv[2 * t] = c < C ? *(const v4f*)hp : v4f{0.f, 0.f, 0.f, 0.f};
          hv[2 * t + 1] = c < C ? *(const v4f*)(hp + 4) : v4f{0.f, 0.f, 0.f, 0.f};
        }
        float s = acc[j];
#pragma unroll
        for (int t = 0; t < kHeadLoads; ++t) {
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            s = fmaf(__uint_as_float((uint32_t)q[t][u] << 16), hv[2 * t + u / 2][2 * (u % 2)], s);
            s = fmaf(__uint_as_float((uint32_t)q[t][u] & 0xFFFF0000u), hv[2 * t + u / 2][2 * (u % 2) + 1], s);
          }
        }
        acc[j] = s;
      }
    }
  }
}

// This lane's share of sum_i w[i] * v[i] over i = lane, lane+64, ... < n
// (bf16 weights, fp32 values), eight loads of each issued before the sums.
__device__ __forceinline__ float head_lane_dot(const uint16_t* __restrict__ w,
                                               const float* __restrict__ v, int n, int lane) {
  float s = 0.f;
  for (int i0 = lane; i0 < n; i0 += 8 * 64) {
    uint16_t wq[8];
    float vq[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int i = i0 + t * 64;
      wq[t] = i < n ? w[i] : (uint16_t)0;
      vq[t] = i < n ? v[i] : 0.f;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) s = fmaf(bf16_to_f32(wq[t]), vq[t], s);
  }
  return s;
}

// Two independent lane dots, (w0 . v0 over n0, w1 . v1 over n1), with the
// loads of both issued together (one memory round trip per 512 entries).
__device__ __forceinline__ void head_lane_dot2(const uint16_t* __restrict__ w0,
                                               const float* __restrict__ v0, int n0,
                                               const uint16_t* __restrict__ w1,
                                               const float* __restrict__ v1, int n1, int lane,
                                               float& s0, float& s1) {
  s0 = 0.f;
  s1 = 0.f;
  const int n = max(n0, n1);
  for (int i0 = lane; i0 < n; i0 += 8 * 64) {
    uint16_t wa[8], wb[8];
    float va[8], vb[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const int i = i0 + t * 64;
      wa[t] = i < n0 ? w0[i] : (uint16_t)0;
      va[t] = i < n0 ? v0[i] : 0.f;
      wb[t] = i < n1 ? w1[i] : (uint16_t)0;
      vb[t] = i < n1 ? v1[i] : 0.f;
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      s0 = fmaf(bf16_to_f32(wa[t]), va[t], s0);
      s1 = fmaf(bf16_to_f32(wb[t]), vb[t], s1);
    }
  }
}

// load(0) + load(1) + ... + load(rows-1), summed in order, eight loads
// issued at a time.
template <typename Load>
__device__ __forceinline__ float head_col_sum(int rows, Load load) {
  float s = 0.f;
  int r = 0;
  for (; r + 8 <= rows; r += 8) {
    float v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = load(r + t);
#pragma unroll
    for (int t = 0; t < 8; ++t) s += v[t];
  }
  for (; r < rows; ++r) s += load(r);
  return s;
}

// f[i][c] = (1/group) * sum over rows [i*group, (i+1)*group) of x[row][c],
// i < n, written to LDS by one 256-thread workgroup: 16-byte loads of 8 rows
// at a time, each column summed over its rows in order (the same arithmetic,
// column by column, as head_col_sum).  C * sizeof(ActT) is a multiple of 16
// and x is 16-byte aligned.  The caller synchronises before reading f.
constexpr int kFusedPoolFloats = 16384;  // pooled rows kept in LDS: 64 KB

template <typename ActT>
__device__ __forceinline__ void head_pool_rows_lds(const ActT* __restrict__ x, int C, int n, int group,
                                                   float* f) {
  constexpr int VW = 16 / sizeof(ActT);  // columns per 16-byte load
  const int nv = C / VW;
  for (int q = threadIdx.x; q < n * nv; q += 256) {
    const int i = q / nv, c = (q - i * nv) * VW;
    float s[VW];
#pragma unroll
    for (int u = 0; u < VW; ++u) s[u] = 0.f;
    for (int r = 0; r < group; r += 8) {
      const int rn = min(8, group - r);
      v4i v[8];
#pragma unroll
      for (int t = 0; t < 8; ++t)
        v[t] = t < rn ? ld16(x + (size_t)(i * group + r + t) * C + c) : zero16();
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        if (t < rn) {
#pragma unroll
          for (int u = 0; u < VW; ++u) {
            float a;
            if constexpr (sizeof(ActT) == 2)
              a = __uint_as_float(((uint32_t)v[t][u / 2] >> (16 * (u % 2))) << 16);
            else
              a = __int_as_float(v[t][u]);
            s[u] += a;
          }
        }
      }
    }
#pragma unroll
    for (int u = 0; u < VW; ++u) f[(size_t)i * C + c + u] = s[u] / (float)group;
  }
}

// Whether a call of n pooled rows of C activations at x may pool inside its
// first layer's kernel (head_pool_rows_lds): few rows, 16-byte loads.
inline bool head_fused_pool_ok(const void* x, int n, int C, size_t act_bytes, int max_groups) {
  return n <= max_groups && (size_t)n * C <= (size_t)kFusedPoolFloats && (C * act_bytes) % 16 == 0 &&
         (uintptr_t)x % 16 == 0;
}

}  // namespace mira
