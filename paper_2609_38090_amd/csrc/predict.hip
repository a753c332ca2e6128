// Predictor head (paper section IV-E): mean-pool a group of token rows of
// layer l's hidden states, then a two-layer MLP (ReLU, sigmoid) scoring the
// experts of layer l+2.  Three small kernels, fp32 accumulation; with few
// pooled rows the pooling runs inside the first layer's kernel.
#include "device_util.h"
#include "head_dev.h"
#include "mira_internal.h"

namespace mira {

// f[i][c] = (1/group) * sum over rows [i*group, (i+1)*group) of x[row][c]
template <typename ActT>
__global__ __launch_bounds__(256) void pred_pool_kernel(const ActT* __restrict__ x, int C, int group,
                                                        float* __restrict__ f) {
  const int i = blockIdx.y;
  const int c = blockIdx.x * 256 + threadIdx.x;
  if (c >= C) return;
  const float s = head_col_sum(group, [&](int r) { return load_act(x, (size_t)(i * group + r) * C + c); });
  f[(size_t)i * C + c] = s / (float)group;
}

// z[i][p] = max(0, sum_c W1[p][c] f[i][c] + b1[p]); one wave per row p, which
// sweeps the row once per kPredGroups pooled rows.
constexpr int kPredGroups = 4;

__global__ __launch_bounds__(256) void pred_layer1_kernel(const uint16_t* __restrict__ w1,
                                                          const float* __restrict__ b1,
                                                          const float* __restrict__ f, int C, int P,
                                                          int n, float* __restrict__ z) {
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (p >= P) return;
  const uint16_t* wr = w1 + (size_t)p * C;
  const float bias = b1 ? b1[p] : 0.f;
  for (int i0 = 0; i0 < n; i0 += kPredGroups) {
    const int ng = min(kPredGroups, n - i0);
    float acc[kPredGroups];
#pragma unroll
    for (int j = 0; j < kPredGroups; ++j) acc[j] = 0.f;
    head_row_dot(wr, f + (size_t)i0 * C, C, ng, lane, acc);
#pragma unroll
    for (int j = 0; j < kPredGroups; ++j) {
      if (j < ng) {
        const float s = wave_sum(acc[j]);
        if (lane == 0) z[(size_t)(i0 + j) * P + p] = fmaxf(s + bias, 0.f);
      }
    }
  }
}

// Pooling and the first layer in one launch, for calls with few pooled rows
// (head_fused_pool_ok): every workgroup pools the n groups into LDS itself,
// so no pooled rows travel through memory and no launch sits between the two
// steps; the results are the same bits as the separate kernels'.
template <typename ActT>
__global__ __launch_bounds__(256) void pred_pool_layer1_kernel(const ActT* __restrict__ x,
                                                               const uint16_t* __restrict__ w1,
                                                               const float* __restrict__ b1, int C,
                                                               int P, int n, int group,
                                                               float* __restrict__ z) {
  extern __shared__ __attribute__((aligned(16))) float f_s[];  // [n][C]
  head_pool_rows_lds(x, C, n, group, f_s);
  __syncthreads();
  const int p = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (p >= P) return;
  float acc[kPredGroups];
#pragma unroll
  for (int j = 0; j < kPredGroups; ++j) acc[j] = 0.f;
  head_row_dot(w1 + (size_t)p * C, f_s, C, n, lane, acc);
  const float bias = b1 ? b1[p] : 0.f;
#pragma unroll
  for (int j = 0; j < kPredGroups; ++j) {
    if (j < n) {
      const float s = wave_sum(acc[j]);
      if (lane == 0) z[(size_t)j * P + p] = fmaxf(s + bias, 0.f);
    }
  }
}

// scores[i][e] = 1 / (1 + exp(-(sum_p W2[e][p] z[i][p] + b2[e]))); one wave per (i, e)
__global__ __launch_bounds__(256) void pred_layer2_kernel(const uint16_t* __restrict__ w2,
                                                          const float* __restrict__ b2,
                                                          const float* __restrict__ z, int P, int E,
                                                          int n, float* __restrict__ scores) {
  const int q = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (q >= n * E) return;
  const int i = q / E, e = q - i * E;
  const uint16_t* wr = w2 + (size_t)e * P;
  const float* zi = z + (size_t)i * P;
  const float s = wave_sum(head_lane_dot(wr, zi, P, lane));
  if (lane == 0) scores[(size_t)i * E + e] = 1.f / (1.f + expf(-(s + (b2 ? b2[e] : 0.f))));
}

hipError_t launch_predict(const mira_pred_shape& p, const void* x, int T, const void* w1,
                          const float* b1, const void* w2, const float* b2, float* scores,
                          void* ws, hipStream_t st) {
  const int n = T / p.group;
  if (n == 0) return hipSuccess;
  float* f = (float*)ws;
  float* z = (float*)((char*)ws + align_up((size_t)n * p.hidden * 4, 256));
  prof_begin("predict", st);
  if (head_fused_pool_ok(x, n, p.hidden, p.act_dtype == MIRA_BF16 ? 2 : 4, kPredGroups)) {
    const size_t lds = (size_t)n * p.hidden * sizeof(float);
    if (p.act_dtype == MIRA_BF16)
      hipLaunchKernelGGL(pred_pool_layer1_kernel<uint16_t>, dim3((p.pred_hidden + 3) / 4), dim3(256), lds,
                         st, (const uint16_t*)x, (const uint16_t*)w1, b1, p.hidden, p.pred_hidden, n,
                         p.group, z);
    else
      hipLaunchKernelGGL(pred_pool_layer1_kernel<float>, dim3((p.pred_hidden + 3) / 4), dim3(256), lds, st,
                         (const float*)x, (const uint16_t*)w1, b1, p.hidden, p.pred_hidden, n, p.group, z);
    hipLaunchKernelGGL(pred_layer2_kernel, dim3((n * p.n_out + 3) / 4), dim3(256), 0, st,
                       (const uint16_t*)w2, b2, z, p.pred_hidden, p.n_out, n, scores);
    prof_end("predict", st);
    return hipGetLastError();
  }
  dim3 gpool((p.hidden + 255) / 256, n);
  if (p.act_dtype == MIRA_BF16)
    hipLaunchKernelGGL(pred_pool_kernel<uint16_t>, gpool, dim3(256), 0, st, (const uint16_t*)x,
                       p.hidden, p.group, f);
  else
    hipLaunchKernelGGL(pred_pool_kernel<float>, gpool, dim3(256), 0, st, (const float*)x, p.hidden,
                       p.group, f);
  hipLaunchKernelGGL(pred_layer1_kernel, dim3((p.pred_hidden + 3) / 4), dim3(256), 0, st,
                     (const uint16_t*)w1, b1, f, p.hidden, p.pred_hidden, n, z);
  hipLaunchKernelGGL(pred_layer2_kernel, dim3((n * p.n_out + 3) / 4), dim3(256), 0, st,
                     (const uint16_t*)w2, b2, z, p.pred_hidden, p.n_out, n, scores);
  prof_end("predict", st);
  return hipGetLastError();
}

}  // namespace mira
