// MixtureHead predictor (paper section IV-E): an ActHead over the pooled
// hidden row and the mean router logits, a HistHead over the selection
// histogram and the top-m indicator, mixed by a contextual gate.  Three
// kernels over all groups of a call: features, the hidden layers of both heads
// plus the gate unit, then the output layers, the mix and the softmax; with
// few groups the features are built inside the hidden layer's kernel.
// fp32 accumulation throughout.
#include "device_util.h"
#include "head_dev.h"
#include "mira_internal.h"

namespace mira {

namespace {

constexpr int kMixGroups = 4;  // groups sharing one pass over a weight row

struct MixWs {
  float* h;     // [n][C] pooled hidden rows
  float* feat;  // [n][3][E] mean logits l, histogram q, top-m indicator u
  float* z;     // [n][Pa + Ph + 1] ReLU'd ActHead and HistHead hidden, gate pre-activation
};

__host__ __device__ inline size_t mix_h_bytes(int n, int C) { return align_up((size_t)n * C * 4, 256); }
__host__ __device__ inline size_t mix_f_bytes(int n, int E) { return align_up((size_t)n * 3 * E * 4, 256); }
__host__ __device__ inline size_t mix_z_bytes(int n, int Pa, int Ph) {
  return align_up((size_t)n * (Pa + Ph + 1) * 4, 256);
}

MixWs mix_ws(void* ws, int n, int C, int E) {
  char* p = (char*)ws;
  MixWs w;
  w.h = (float*)p;
  w.feat = (float*)(p + mix_h_bytes(n, C));
  w.z = (float*)(p + mix_h_bytes(n, C) + mix_f_bytes(n, E));
  return w;
}

// Routing features of group i, by one 256-thread workgroup: fi[0..E) the
// mean router logits, fi[E..2E) the selection histogram (share of the
// group's pairs per expert), fi[2E..3E) the indicator of the m most selected
// experts (ties to the lower index).  cnt is E ints of LDS.
__device__ __forceinline__ void group_features(const float* __restrict__ logits,
                                               const int32_t* __restrict__ topk_idx, int E, int k,
                                               int m, int group, int i, int* cnt, float* fi) {
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += 256) cnt[e] = 0;
  __syncthreads();
  const int pairs = group * k;
  const int32_t* ti = topk_idx + (size_t)i * pairs;
  for (int p = tid; p < pairs; p += 256) {
    const int e = ti[p];
    if (e >= 0 && e < E) atomicAdd(&cnt[e], 1);
  }
  __syncthreads();
  for (int e = tid; e < E; e += 256) {
    const float s = head_col_sum(group, [&](int r) { return logits[(size_t)(i * group + r) * E + e]; });
    const int c = cnt[e];
    int rank = 0;  // experts ahead of e: more pairs, or as many and a lower index
    for (int f = 0; f < E; ++f) rank += (cnt[f] > c) || (cnt[f] == c && f < e);
    fi[e] = s / (float)group;
    fi[E + e] = (float)c / (float)pairs;
    fi[2 * E + e] = (rank < m && c > 0) ? 1.f : 0.f;
  }
}

// Grid (C/256 + 1, n).  Blocks x < C/256 pool 256 hidden columns of group
// blockIdx.y; the last block builds the routing features of that group.
template <typename ActT>
__global__ __launch_bounds__(256) void mix_features_kernel(const ActT* __restrict__ x,
                                                           const float* __restrict__ logits,
                                                           const int32_t* __restrict__ topk_idx,
                                                           int C, int E, int k, int m, int group,
                                                           float* __restrict__ h,
                                                           float* __restrict__ feat) {
  const int i = blockIdx.y, tid = threadIdx.x;
  const int ncb = (C + 255) / 256;
  if ((int)blockIdx.x < ncb) {
    const int c = blockIdx.x * 256 + tid;
    if (c >= C) return;
    const float s = head_col_sum(group, [&](int r) { return load_act(x, (size_t)(i * group + r) * C + c); });
    h[(size_t)i * C + c] = s / (float)group;
    return;
  }
  __shared__ int cnt[MIRA_MAX_EXPERTS];
  group_features(logits, topk_idx, E, k, m, group, i, cnt, feat + (size_t)i * 3 * E);
}

// Row r of the stacked hidden layer, by one wave: rows [0, Pa) are the
// ActHead, [Pa, Pa+Ph) the HistHead, row Pa+Ph the gate unit.  The wave
// sweeps its weight row once per kMixGroups groups.
__device__ __forceinline__ void hidden_row(const mira_mixture_weights& w, int C, int E, int Pa, int Ph,
                                           int n, const float* h, const float* feat,
                                           float* __restrict__ z, int r, int lane) {
  const int rows = Pa + Ph + 1;
  const uint16_t *wc = nullptr, *wl = nullptr, *wq = nullptr, *wu = nullptr;
  float bias = 0.f;
  bool relu = true;
  if (r < Pa) {
    wc = (const uint16_t*)w.wah + (size_t)r * C;
    wl = (const uint16_t*)w.wal + (size_t)r * E;
    bias = w.ba1 ? w.ba1[r] : 0.f;
  } else if (r < Pa + Ph) {
    const int p = r - Pa;
    wq = (const uint16_t*)w.whq + (size_t)p * E;
    wu = (const uint16_t*)w.whu + (size_t)p * E;
    bias = w.bh1 ? w.bh1[p] : 0.f;
  } else {
    wc = (const uint16_t*)w.gh;
    wl = (const uint16_t*)w.gl;
    wq = (const uint16_t*)w.gq;
    wu = (const uint16_t*)w.gu;
    bias = w.bg;
    relu = false;
  }
  for (int i0 = 0; i0 < n; i0 += kMixGroups) {
    const int ng = min(kMixGroups, n - i0);
    float acc[kMixGroups];
#pragma unroll
    for (int j = 0; j < kMixGroups; ++j) acc[j] = 0.f;
    if (wc) head_row_dot(wc, h + (size_t)i0 * C, C, ng, lane, acc);
#pragma unroll
    for (int j = 0; j < kMixGroups; ++j) {
      if (j < ng) {
        const float* fi = feat + (size_t)(i0 + j) * 3 * E;
        float s = acc[j];
        if (wl) s += head_lane_dot(wl, fi, E, lane);
        if (wq) s += head_lane_dot(wq, fi + E, E, lane);
        if (wu) s += head_lane_dot(wu, fi + 2 * E, E, lane);
        s = wave_sum(s) + bias;
        if (lane == 0) z[(size_t)(i0 + j) * rows + r] = relu ? fmaxf(s, 0.f) : s;
      }
    }
  }
}

// One wave per row of the stacked hidden layer (hidden_row).
__global__ __launch_bounds__(256) void mix_hidden_kernel(mira_mixture_weights w, int C, int E,
                                                         int Pa, int Ph, int n,
                                                         const float* __restrict__ h,
                                                         const float* __restrict__ feat,
                                                         float* __restrict__ z) {
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= Pa + Ph + 1) return;
  hidden_row(w, C, E, Pa, Ph, n, h, feat, z, r, lane);
}

// Features and the hidden layer in one launch, for calls with few groups
// (head_fused_pool_ok and the features in LDS): every workgroup pools the
// hidden rows and builds the routing features of all groups in LDS itself,
// with the arithmetic of the separate kernels, so the bits are the same.
template <typename ActT>
__global__ __launch_bounds__(256) void mix_fused_hidden_kernel(const ActT* __restrict__ x,
                                                               const float* __restrict__ logits,
                                                               const int32_t* __restrict__ topk_idx,
                                                               mira_mixture_weights w, int C, int E,
                                                               int k, int m, int group, int Pa, int Ph,
                                                               int n, float* __restrict__ z) {
  extern __shared__ __attribute__((aligned(16))) float sm[];  // [n][C] pooled, then [n][3][E]
  __shared__ int cnt[MIRA_MAX_EXPERTS];
  float* h_s = sm;
  float* f_s = sm + (size_t)n * C;
  head_pool_rows_lds(x, C, n, group, h_s);
  for (int i = 0; i < n; ++i) {
    group_features(logits, topk_idx, E, k, m, group, i, cnt, f_s + (size_t)i * 3 * E);
    __syncthreads();  // cnt is reused by the next group
  }
  const int r = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (r >= Pa + Ph + 1) return;
  hidden_row(w, C, E, Pa, Ph, n, h_s, f_s, z, r, lane);
}

// One block of 16 waves per group: a wave per output (both output layers'
// dots issued together), the gate, the mix and the softmax.
constexpr int kOutWaves = 16;

__global__ __launch_bounds__(kOutWaves * 64) void mix_out_kernel(mira_mixture_weights w, int Pa,
                                                                 int Ph, int N,
                                                                 const float* __restrict__ z,
                                                                 float* __restrict__ probs,
                                                                 float* __restrict__ alpha_out) {
  __shared__ float ys[MIRA_MAX_EXPERTS];
  __shared__ float red[kOutWaves];
  const int i = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int rows = Pa + Ph + 1;
  const float* zi = z + (size_t)i * rows;
  const float alpha = 1.f / (1.f + expf(-zi[Pa + Ph]));
  for (int e = wave; e < N; e += kOutWaves) {
    float a, b;
    head_lane_dot2((const uint16_t*)w.wa2 + (size_t)e * Pa, zi, Pa,
                   (const uint16_t*)w.wh2 + (size_t)e * Ph, zi + Pa, Ph, lane, a, b);
    a = wave_sum(a) + (w.ba2 ? w.ba2[e] : 0.f);
    b = wave_sum(b) + (w.bh2 ? w.bh2[e] : 0.f);
    if (lane == 0) ys[e] = alpha * a + (1.f - alpha) * b;
  }
  __syncthreads();
  // softmax over the N mixed logits, N <= 256: thread e < N holds ys[e]
  const float y = tid < N ? ys[tid] : -__builtin_inff();
  float v = wave_max(y);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float ymax = red[0];
  for (int q = 1; q < kOutWaves; ++q) ymax = fmaxf(ymax, red[q]);
  __syncthreads();
  const float ex = tid < N ? expf(y - ymax) : 0.f;
  v = wave_sum(ex);
  if (lane == 0) red[wave] = v;
  __syncthreads();
  float denom = 0.f;
  for (int q = 0; q < kOutWaves; ++q) denom += red[q];
  if (tid < N) probs[(size_t)i * N + tid] = ex / denom;
  if (tid == 0 && alpha_out) alpha_out[i] = alpha;
}

}  // namespace

size_t mixture_ws_bytes(int n, const mira_mixture_shape& p) {
  return mix_h_bytes(n, p.hidden) + mix_f_bytes(n, p.n_src) +
         mix_z_bytes(n, p.act_hidden, p.hist_hidden);
}

hipError_t launch_mixture(const mira_mixture_shape& p, const mira_mixture_weights& w,
                          const void* x, const float* logits, const int32_t* topk_idx, int T,
                          float* probs, float* alpha, void* ws, hipStream_t st) {
  const int n = T / p.group;
  if (n == 0) return hipSuccess;
  const int C = p.hidden, E = p.n_src, Pa = p.act_hidden, Ph = p.hist_hidden;
  const MixWs m = mix_ws(ws, n, C, E);
  prof_begin("mixture", st);
  const size_t fused_floats = (size_t)n * C + (size_t)n * 3 * E;
  if (head_fused_pool_ok(x, n, C, p.act_dtype == MIRA_BF16 ? 2 : 4, kMixGroups) &&
      fused_floats <= (size_t)kFusedPoolFloats) {
    const dim3 gh((Pa + Ph + 1 + 3) / 4);
    const size_t lds = fused_floats * sizeof(float);
    if (p.act_dtype == MIRA_BF16)
      hipLaunchKernelGGL(mix_fused_hidden_kernel<uint16_t>, gh, dim3(256), lds, st, (const uint16_t*)x, logits,
                         topk_idx, w, C, E, p.top_k, p.hist_top, p.group, Pa, Ph, n, m.z);
    else
      hipLaunchKernelGGL(mix_fused_hidden_kernel<float>, gh, dim3(256), lds, st, (const float*)x, logits,
                         topk_idx, w, C, E, p.top_k, p.hist_top, p.group, Pa, Ph, n, m.z);
  } else {
    const dim3 gf((C + 255) / 256 + 1, n);
    if (p.act_dtype == MIRA_BF16)
      hipLaunchKernelGGL(mix_features_kernel<uint16_t>, gf, dim3(256), 0, st, (const uint16_t*)x,
                         logits, topk_idx, C, E, p.top_k, p.hist_top, p.group, m.h, m.feat);
    else
      hipLaunchKernelGGL(mix_features_kernel<float>, gf, dim3(256), 0, st, (const float*)x, logits,
                         topk_idx, C, E, p.top_k, p.hist_top, p.group, m.h, m.feat);
    hipLaunchKernelGGL(mix_hidden_kernel, dim3((Pa + Ph + 1 + 3) / 4), dim3(256), 0, st, w, C, E, Pa,
                       Ph, n, m.h, m.feat, m.z);
  }
  hipLaunchKernelGGL(mix_out_kernel, dim3(n), dim3(kOutWaves * 64), 0, st, w, Pa, Ph, p.n_out, m.z, probs,
                     alpha);
  prof_end("mixture", st);
  return hipGetLastError();
}

}  // namespace mira
