// Router logits, top-k selection, combine weights and the stable
// token-to-expert permutation (paper section II-A: the router scores every
// expert for each token, the top-k experts process it, their outputs are
// combined).
//
// Two launch shapes share the device functions below:
//  - prefill: route_kernel (16 tokens per workgroup) then permute_kernel
//    (one workgroup);
//  - decode (T <= MIRA_DECODE_MAX_TOKENS): one workgroup runs router, top-k,
//    permutation and the fixed-point digits of x back to back, so the
//    expert kernels start after a single small launch.
#include "device_util.h"
#include "mira_internal.h"

namespace mira {

constexpr int kRouteTok = 16;  // tokens per route workgroup
constexpr int kRouteThreads = 256;
constexpr int kBigThreads = 1024;  // permutation and decode-prep workgroups
constexpr int kBigWaves = kBigThreads / 64;

// ---------------------------------------------------------------------------
// Router logits for 16 tokens: lg[t][e] = sum_c x[t][c] * Wg[e][c] + b[e].
// bf16: MFMA, A = Wg rows (experts), B = x rows (tokens), fp32 accumulate;
// waves split the expert tiles.  fp32: VALU dot products, fp32 accumulate.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void logits_tile_bf16(const uint16_t* __restrict__ x,
                                                 const uint16_t* __restrict__ wr,
                                                 const float* __restrict__ bias, int T, int E,
                                                 int C, int t0, int nwaves,
                                                 float (*lg)[MIRA_MAX_EXPERTS]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int n_et = (E + 15) / 16;
  const int t = t0 + r16;
  const bool tok_ok = t < T;
  const uint16_t* xrow = x + (size_t)(tok_ok ? t : 0) * C + kg * 8;
  for (int et = wave; et < n_et; et += nwaves) {
    const int e = et * 16 + r16;
    const bool e_ok = e < E;
    const uint16_t* wrow = wr + (size_t)(e_ok ? e : 0) * C + kg * 8;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    int k0 = 0;
    for (; k0 + 128 <= C; k0 += 128) {
      v4i a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = e_ok ? ld16(wrow + k0 + 32 * u) : zero16();
        b[u] = tok_ok ? ld16(xrow + k0 + 32 * u) : zero16();
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) acc = mfma_bf16(a[u], b[u], acc);
    }
    for (; k0 < C; k0 += 32) {
      v4i a = e_ok ? ld16(wrow + k0) : zero16();
      v4i b = tok_ok ? ld16(xrow + k0) : zero16();
      acc = mfma_bf16(a, b, acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {  // D[expert 4*kg+i][token r16]
      const int ee = et * 16 + kg * 4 + i;
      if (ee < E) lg[r16][ee] = acc[i] + (bias ? bias[ee] : 0.f);
    }
  }
}

__device__ __forceinline__ void logits_tile_f32(const float* __restrict__ x,
                                                const float* __restrict__ wr,
                                                const float* __restrict__ bias, int T, int E,
                                                int C, int t0, int nwaves,
                                                float (*lg)[MIRA_MAX_EXPERTS]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ntok = min(kRouteTok, T - t0);
  for (int pr = wave; pr < ntok * E; pr += nwaves) {
    const int tt = pr / E, e = pr - tt * E;
    const float* xr = x + (size_t)(t0 + tt) * C;
    const float* wrow = wr + (size_t)e * C;
    float s = 0.f;
    for (int c = lane; c < C; c += 64) s = fmaf(xr[c], wrow[c], s);
    s = wave_sum(s);
    if (lane == 0) lg[tt][e] = s + (bias ? bias[e] : 0.f);
  }
}

// Decode variant for bf16: all waves of the workgroup split the k range of
// every expert tile; partial sums are reduced through LDS in wave order.
__device__ void logits_ksplit_bf16(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wr,
                                   const float* __restrict__ bias, int T, int E, int C,
                                   float (*part)[16][17], float (*lg)[MIRA_MAX_EXPERTS]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int n_et = (E + 15) / 16, nch = C / 32;
  const bool tok_ok = r16 < T;
  const uint16_t* xrow = x + (size_t)(tok_ok ? r16 : 0) * C + kg * 8;
  for (int et = 0; et < n_et; ++et) {
    const int e = et * 16 + r16;
    const bool e_ok = e < E;
    const uint16_t* wrow = wr + (size_t)(e_ok ? e : 0) * C + kg * 8;
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    int ch = wave;
    for (; ch + 3 * kBigWaves < nch; ch += 4 * kBigWaves) {
      v4i a[4], b[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        a[u] = e_ok ? ld16(wrow + (ch + u * kBigWaves) * 32) : zero16();
        b[u] = tok_ok ? ld16(xrow + (ch + u * kBigWaves) * 32) : zero16();
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) acc = mfma_bf16(a[u], b[u], acc);
    }
    for (; ch < nch; ch += kBigWaves) {
      v4i a = e_ok ? ld16(wrow + ch * 32) : zero16();
      v4i b = tok_ok ? ld16(xrow + ch * 32) : zero16();
      acc = mfma_bf16(a, b, acc);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) part[wave][r16][kg * 4 + i] = acc[i];  // [token][expert]
    __syncthreads();
    if (tid < 256) {
      const int tt = tid >> 4, ee = tid & 15, e2 = et * 16 + ee;
      float s = 0.f;
      for (int w = 0; w < kBigWaves; ++w) s += part[w][tt][ee];
      if (e2 < E) lg[tt][e2] = s + (bias ? bias[e2] : 0.f);
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Top-k of one token (one wave): repeatedly take the largest key (value,
// then the lower index), then the combine weights.  Lanes j < k write
// selection j.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void topk_token(const float* __restrict__ lgrow, int E, int k,
                                           int softmax_all, int32_t* idx_a, float* w_a,
                                           int32_t* idx_b, float* w_b) {
  const int lane = threadIdx.x & 63;
  uint32_t khi[MIRA_MAX_EXPERTS / 64], klo[MIRA_MAX_EXPERTS / 64];
#pragma unroll
  for (int i = 0; i < MIRA_MAX_EXPERTS / 64; ++i) {
    const int e = lane + 64 * i;
    khi[i] = e < E ? f32_order_key(lgrow[e]) : 0u;
    klo[i] = e < E ? ~(uint32_t)e : 0u;
  }
  int my_e = 0;
  float my_v = 0.f;
  for (int j = 0; j < k; ++j) {
    uint32_t bh = 0, bl = 0;
#pragma unroll
    for (int i = 0; i < MIRA_MAX_EXPERTS / 64; ++i)
      if (khi[i] > bh || (khi[i] == bh && klo[i] > bl)) {
        bh = khi[i];
        bl = klo[i];
      }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      const uint32_t oh = __shfl_xor(bh, o, 64), ol = __shfl_xor(bl, o, 64);
      if (oh > bh || (oh == bh && ol > bl)) {
        bh = oh;
        bl = ol;
      }
    }
    const int e_sel = (int)~bl;
    if (lane == j) {
      my_e = e_sel;
      my_v = lgrow[e_sel];
    }
    if (lane == (e_sel & 63)) {
#pragma unroll
      for (int i = 0; i < MIRA_MAX_EXPERTS / 64; ++i)
        if (i == (e_sel >> 6)) khi[i] = klo[i] = 0u;
    }
  }
  const float vmax = __shfl(my_v, 0, 64);
  const float ex = lane < k ? expf(my_v - vmax) : 0.f;
  float denom;
  if (softmax_all) {
    float s = 0.f;
    for (int e = lane; e < E; e += 64) s += expf(lgrow[e] - vmax);
    denom = wave_sum(s);
  } else {
    denom = wave_sum(ex);
  }
  if (lane < k) {
    const float w = ex / denom;
    idx_a[lane] = my_e;
    w_a[lane] = w;
    if (idx_b) idx_b[lane] = my_e;
    if (w_b) w_b[lane] = w;
  }
}

template <typename ActT>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(
    const ActT* __restrict__ x, const ActT* __restrict__ wr, const float* __restrict__ bias,
    int T, int E, int C, int k, int softmax_all, float* __restrict__ logits_ws,
    float* __restrict__ logits_out, int32_t* __restrict__ idx_ws, float* __restrict__ w_ws) {
  __shared__ float lg[kRouteTok][MIRA_MAX_EXPERTS];
  const int t0 = blockIdx.x * kRouteTok;
  if constexpr (sizeof(ActT) == 2)
    logits_tile_bf16(x, wr, bias, T, E, C, t0, kRouteThreads / 64, lg);
  else
    logits_tile_f32(x, wr, bias, T, E, C, t0, kRouteThreads / 64, lg);
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int tt = wave; tt < kRouteTok; tt += kRouteThreads / 64) {
    const int t = t0 + tt;
    if (t >= T) break;
    for (int e = lane; e < E; e += 64) {
      logits_ws[(size_t)t * E + e] = lg[tt][e];
      if (logits_out) logits_out[(size_t)t * E + e] = lg[tt][e];
    }
    topk_token(lg[tt], E, k, softmax_all, idx_ws + (size_t)t * k, w_ws + (size_t)t * k, nullptr,
               nullptr);
  }
}

// ---------------------------------------------------------------------------
// Stable grouping of (token, slot) pairs by expert (one 1024-thread
// workgroup).  Routed pair p = t*k + j goes to expert idx[p]; shared expert s
// owns pairs T*k + s*T + t.  Groups: routed experts 0..E-1 then shared
// 0..S-1; inside a group pairs keep increasing p.  Outputs: counts, offsets,
// inv[p] = position, tokpos/wpos (token and combine weight at each position),
// the list of non-empty groups, the prefill m-tile prefix, and residency
// status bits.  Ranks come from wave ballots, never from the order of
// atomics, so the result is deterministic.  idx and wts may point to LDS or
// global memory.
// ---------------------------------------------------------------------------
struct PermOut {
  int32_t* counts_ws;
  int32_t* offsets;
  int32_t* inv;
  int32_t* tokpos;
  float* wpos;
  int32_t* misc;
  int32_t* active;
  int32_t* mstart;
  int32_t* counts_out;
  int32_t* idx_out;
  float* w_out;
  int32_t* offsets_out;
  int32_t* order_out;
};

__device__ void permute_body(const int32_t* idx, const float* wts, int T, int k, int E, int S,
                             int BM, const ExpertPool& ep, const PermOut& o) {
  __shared__ int hist[kBigWaves][MIRA_MAX_EXPERTS];
  __shared__ int off_s[MIRA_MAX_EXPERTS + 1];
  __shared__ int mst_s[MIRA_MAX_EXPERTS + 1];
  __shared__ int act_s[MIRA_MAX_EXPERTS];
  __shared__ int n_act_s;
  __shared__ int status_s;
  const int G = E + S, Tk = T * k;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  for (int i = tid; i < kBigWaves * MIRA_MAX_EXPERTS; i += kBigThreads) (&hist[0][0])[i] = 0;
  if (tid == 0) status_s = 0;
  __syncthreads();

  // pass 1: per-wave histograms over contiguous ranges of routed pairs
  const int span = (Tk + kBigWaves - 1) / kBigWaves;
  const int p_beg = wave * span, p_end = min(Tk, p_beg + span);
  for (int p = p_beg + lane; p < p_end; p += 64) {
    const int e = idx[p];
    atomicAdd(&hist[wave][e], 1);
    if (o.idx_out) o.idx_out[p] = e;
    if (o.w_out) o.w_out[p] = wts[p];
  }
  __syncthreads();

  // counts and exclusive scan (wave 0: each lane owns 4 consecutive groups)
  if (wave == 0) {
    int c4[4], sum = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = lane * 4 + i;
      int c = 0;
      if (g < E) {
        for (int w = 0; w < kBigWaves; ++w) c += hist[w][g];
      } else if (g < G) {
        c = T;
      }
      c4[i] = c;
      sum += c;
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off, 64);
      if (lane >= off) incl += v;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = lane * 4 + i;
      if (g < G) {
        off_s[g] = run;
        o.counts_ws[g] = c4[i];
        if (o.counts_out) o.counts_out[g] = c4[i];
      }
      run += c4[i];
    }
    if (lane == 63) off_s[G] = incl;
  }
  __syncthreads();
  for (int g = tid; g <= G; g += kBigThreads) {
    o.offsets[g] = off_s[g];
    if (o.offsets_out) o.offsets_out[g] = off_s[g];
  }
  // per-wave bases: offset of the group plus pairs of earlier waves
  for (int g = tid; g < E; g += kBigThreads) {
    int b = off_s[g];
    for (int w = 0; w < kBigWaves; ++w) {
      const int c = hist[w][g];
      hist[w][g] = b;
      b += c;
    }
  }
  __syncthreads();

  // pass 2: stable scatter; ranks within a 64-pair chunk from ballots
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int base = p_beg; base < p_end; base += 64) {
    const int p = base + lane;
    const bool ok = p < p_end;
    const int e = ok ? idx[p] : 0;
    uint64_t same = __ballot(ok);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t b = __ballot(ok && ((e >> bit) & 1));
      same &= ((e >> bit) & 1) ? b : ~b;
    }
    const int rank = __popcll(same & lt_mask);
    int b0 = 0;
    if (ok) b0 = hist[wave][e];
    const bool leader = ok && (same & lt_mask) == 0;
    __builtin_amdgcn_wave_barrier();  // every lane has read its base
    if (ok) {
      const int pos = b0 + rank;
      o.inv[p] = pos;
      o.tokpos[pos] = p / k;
      o.wpos[pos] = wts[p];
      if (o.order_out) o.order_out[pos] = p;
    }
    if (leader) hist[wave][e] = b0 + __popcll(same);
    __builtin_amdgcn_wave_barrier();
  }
  // shared experts: every token, in token order, weight 1
  for (int i = tid; i < S * T; i += kBigThreads) {
    const int s = i / T, t = i - s * T;
    const int pos = off_s[E + s] + t;
    o.inv[Tk + i] = pos;
    o.tokpos[pos] = t;
    o.wpos[pos] = 1.0f;
    if (o.order_out) o.order_out[pos] = Tk + i;
  }

  // non-empty groups, residency status, prefill m-tiles
  if (wave == 0) {
    int cnt4[4], mt4[4], na = 0, nm = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = lane * 4 + i;
      const int c = g < G ? off_s[g + 1] - off_s[g] : 0;
      cnt4[i] = c;
      mt4[i] = (c + BM - 1) / BM;
      na += c > 0;
      nm += mt4[i];
    }
    int ia = na, im = nm;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int va = __shfl_up(ia, off, 64), vm = __shfl_up(im, off, 64);
      if (lane >= off) {
        ia += va;
        im += vm;
      }
    }
    int ra = ia - na, rm = im - nm, bits = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = lane * 4 + i;
      if (g < G) {
        mst_s[g] = rm;
        if (cnt4[i] > 0) {
          act_s[ra++] = g;
          const int slot = ep.slot_table[g];
          if (slot < 0) bits |= 1;
          else if (slot >= ep.n_slots) bits |= 2;
        }
      }
      rm += mt4[i];
    }
    if (lane == 63) {
      n_act_s = ia;
      mst_s[G] = im;
    }
    if (bits) atomicOr(&status_s, bits);
  }
  __syncthreads();
  for (int g = tid; g <= G; g += kBigThreads) o.mstart[g] = mst_s[g];
  for (int a = tid; a < n_act_s; a += kBigThreads) o.active[a] = act_s[a];
  if (tid == 0) {
    o.misc[MISC_NACTIVE] = n_act_s;
    o.misc[MISC_MTOTAL] = mst_s[G];
    if (ep.status) *ep.status = status_s;
  }
}

__global__ __launch_bounds__(kBigThreads) void permute_kernel(const int32_t* __restrict__ idx,
                                                              const float* __restrict__ wts, int T,
                                                              int k, int E, int S, int BM,
                                                              ExpertPool ep, PermOut o) {
  permute_body(idx, wts, T, k, E, S, BM, ep, o);
}

// ---------------------------------------------------------------------------
// Decode preparation (T <= 16 tokens, one workgroup): router logits, top-k
// and weights, permutation, and the fixed-point digits of x used by the
// integer expert kernels (|x * 2^E_t| < 2^22 per token, three signed
// base-256 digits; layout xdig[(t*3 + d)*C + c], xexp[t] = E_t).
// ---------------------------------------------------------------------------
template <typename ActT>
__global__ __launch_bounds__(kBigThreads) void decode_prep_kernel(
    const ActT* __restrict__ x, const ActT* __restrict__ wr, const float* __restrict__ bias,
    int T, int E, int C, int k, int S, int softmax_all, float* __restrict__ logits_out,
    ExpertPool ep, PermOut o, int8_t* __restrict__ xdig, int32_t* __restrict__ xexp) {
  __shared__ float lg[kRouteTok][MIRA_MAX_EXPERTS];
  __shared__ float part[kBigWaves][16][17];
  __shared__ int32_t idx_s[kRouteTok * MIRA_MAX_TOPK];
  __shared__ float w_s[kRouteTok * MIRA_MAX_TOPK];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;

  if constexpr (sizeof(ActT) == 2) {
    logits_ksplit_bf16(x, wr, bias, T, E, C, part, lg);
  } else {
    logits_tile_f32(x, wr, bias, T, E, C, 0, kBigWaves, lg);
    __syncthreads();
  }
  if (wave < T) {
    const int t = wave;
    if (logits_out)
      for (int e = lane; e < E; e += 64) logits_out[(size_t)t * E + e] = lg[t][e];
    topk_token(lg[t], E, k, softmax_all, idx_s + t * k, w_s + t * k, nullptr, nullptr);
  }
  __syncthreads();
  permute_body(idx_s, w_s, T, k, E, S, kPrefBM, ep, o);

  // fixed-point digits of x, one wave per token
  if (wave < T) {
    const int t = wave;
    const ActT* xr = x + (size_t)t * C;
    float m = 0.f;
    for (int c = lane; c < C; c += 64) m = fmaxf(m, fabsf(load_act(xr, c)));
    m = wave_max(m);
    const int Ex = kFixBits - exp_bound(m);
    int8_t* d0p = xdig + (size_t)t * kDigits * C;
    for (int c = lane * 4; c < C; c += 256) {
      uint32_t w0 = 0, w1 = 0, w2 = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int v = (int)rintf(ldexpf(load_act(xr, c + i), Ex));
        int d0, d1, d2;
        split_digits(v, d0, d1, d2);
        w0 |= (uint32_t)(d0 & 0xFF) << (8 * i);
        w1 |= (uint32_t)(d1 & 0xFF) << (8 * i);
        w2 |= (uint32_t)(d2 & 0xFF) << (8 * i);
      }
      *(uint32_t*)(d0p + c) = w0;
      *(uint32_t*)(d0p + C + c) = w1;
      *(uint32_t*)(d0p + 2 * C + c) = w2;
    }
    if (lane == 0) xexp[t] = Ex;
  }
}

static PermOut perm_out(const WsPtr& w, int32_t* counts_out, int32_t* idx_out, float* wts_out,
                        int32_t* offsets_out, int32_t* order_out) {
  PermOut o;
  o.counts_ws = w.counts;
  o.offsets = w.offsets;
  o.inv = w.inv;
  o.tokpos = w.tokpos;
  o.wpos = w.wpos;
  o.misc = w.misc;
  o.active = w.active;
  o.mstart = w.mstart;
  o.counts_out = counts_out;
  o.idx_out = idx_out;
  o.w_out = wts_out;
  o.offsets_out = offsets_out;
  o.order_out = order_out;
  return o;
}

hipError_t launch_route(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                        const void* wr, const float* bias, float* logits_out, hipStream_t st) {
  const int T = L.T;
  if (T == 0) return hipSuccess;
  dim3 grid((T + kRouteTok - 1) / kRouteTok), block(kRouteThreads);
  const int sa = (s.flags & MIRA_FLAG_SOFTMAX_ALL) ? 1 : 0;
  prof_begin("route", st);
  if (s.act_dtype == MIRA_BF16)
    hipLaunchKernelGGL(route_kernel<uint16_t>, grid, block, 0, st, (const uint16_t*)x,
                       (const uint16_t*)wr, bias, T, L.E, L.C, L.k, sa, w.logits, logits_out,
                       w.idx, w.wts);
  else
    hipLaunchKernelGGL(route_kernel<float>, grid, block, 0, st, (const float*)x,
                       (const float*)wr, bias, T, L.E, L.C, L.k, sa, w.logits, logits_out, w.idx,
                       w.wts);
  prof_end("route", st);
  return hipGetLastError();
}

hipError_t launch_permute(const mira_shape& s, const Layout& L, const WsPtr& w,
                          const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                          float* wts_out, int32_t* offsets_out, int32_t* order_out,
                          hipStream_t st) {
  prof_begin("permute", st);
  hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(kBigThreads), 0, st, w.idx, w.wts, L.T, L.k,
                     L.E, L.S, kPrefBM, ep,
                     perm_out(w, counts_out, idx_out, wts_out, offsets_out, order_out));
  prof_end("permute", st);
  return hipGetLastError();
}

hipError_t launch_decode_prep(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                              const void* wr, const float* bias, float* logits_out,
                              const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                              float* wts_out, int32_t* offsets_out, int32_t* order_out,
                              hipStream_t st) {
  if (L.T == 0) return hipSuccess;
  const int sa = (s.flags & MIRA_FLAG_SOFTMAX_ALL) ? 1 : 0;
  const PermOut o = perm_out(w, counts_out, idx_out, wts_out, offsets_out, order_out);
  prof_begin("decode_prep", st);
  if (s.act_dtype == MIRA_BF16)
    hipLaunchKernelGGL(decode_prep_kernel<uint16_t>, dim3(1), dim3(kBigThreads), 0, st,
                       (const uint16_t*)x, (const uint16_t*)wr, bias, L.T, L.E, L.C, L.k, L.S, sa,
                       logits_out, ep, o, w.xdig, w.xexp);
  else
    hipLaunchKernelGGL(decode_prep_kernel<float>, dim3(1), dim3(kBigThreads), 0, st,
                       (const float*)x, (const float*)wr, bias, L.T, L.E, L.C, L.k, L.S, sa,
                       logits_out, ep, o, w.xdig, w.xexp);
  prof_end("decode_prep", st);
  return hipGetLastError();
}

__global__ void set_slot_kernel(int32_t* table, int expert, int slot) { table[expert] = slot; }

hipError_t launch_set_slot(int32_t* table, int expert, int slot, hipStream_t st) {
  hipLaunchKernelGGL(set_slot_kernel, dim3(1), dim3(1), 0, st, table, expert, slot);
  return hipGetLastError();
}

}  // namespace mira
