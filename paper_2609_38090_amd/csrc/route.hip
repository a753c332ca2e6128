// Router logits, top-k selection, combine weights and the stable
// token-to-expert permutation (paper section II-A: the router scores every
// expert for each token, the top-k experts process it, their outputs are
// combined).
#include "device_util.h"
#include "mira_internal.h"

namespace mira {

constexpr int kRouteTok = 16;  // tokens per route workgroup
constexpr int kRouteThreads = 256;

// ---------------------------------------------------------------------------
// Router logits l[t][e] = sum_c x[t][c] * Wg[e][c] + b[e] (fp32 accumulate)
// for 16 tokens per workgroup, then per-token top-k and combine weights.
// bf16 activations use MFMA (exact products, fp32 sums); fp32 ones use VALU.
// ---------------------------------------------------------------------------
template <typename ActT>
__device__ __forceinline__ void route_logits_tile(const ActT* __restrict__ x,
                                                  const ActT* __restrict__ wr,
                                                  const float* __restrict__ bias, int T, int E,
                                                  int C, int t0, float (*lg)[MIRA_MAX_EXPERTS]);

template <>
__device__ __forceinline__ void route_logits_tile<uint16_t>(const uint16_t* __restrict__ x,
                                                            const uint16_t* __restrict__ wr,
                                                            const float* __restrict__ bias, int T,
                                                            int E, int C, int t0,
                                                            float (*lg)[MIRA_MAX_EXPERTS]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int n_et = (E + 15) / 16;
  const int t = t0 + r16;
  const bool tok_ok = t < T;
  const uint16_t* xrow = x + (size_t)(tok_ok ? t : 0) * C + kg * 8;
  for (int et = wave; et < n_et; et += kRouteThreads / 64) {
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
    // D[expert 4*kg+i][token r16]
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int ee = et * 16 + kg * 4 + i;
      if (ee < E) lg[r16][ee] = acc[i] + (bias ? bias[ee] : 0.f);
    }
  }
}

template <>
__device__ __forceinline__ void route_logits_tile<float>(const float* __restrict__ x,
                                                         const float* __restrict__ wr,
                                                         const float* __restrict__ bias, int T,
                                                         int E, int C, int t0,
                                                         float (*lg)[MIRA_MAX_EXPERTS]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int tt = wave; tt < kRouteTok; tt += kRouteThreads / 64) {
    const int t = t0 + tt;
    if (t >= T) break;
    const float* xr = x + (size_t)t * C;
    for (int e = 0; e < E; ++e) {
      const float* wrow = wr + (size_t)e * C;
      float s = 0.f;
      for (int c = lane; c < C; c += 64) s = fmaf(xr[c], wrow[c], s);
      s = wave_sum(s);
      if (lane == 0) lg[tt][e] = s + (bias ? bias[e] : 0.f);
    }
  }
}

template <typename ActT>
__global__ __launch_bounds__(kRouteThreads) void route_kernel(
    const ActT* __restrict__ x, const ActT* __restrict__ wr, const float* __restrict__ bias,
    int T, int E, int C, int k, int softmax_all, float* __restrict__ logits_ws,
    float* __restrict__ logits_out, int32_t* __restrict__ idx_ws, float* __restrict__ w_ws) {
  __shared__ float lg[kRouteTok][MIRA_MAX_EXPERTS];
  const int t0 = blockIdx.x * kRouteTok;
  route_logits_tile<ActT>(x, wr, bias, T, E, C, t0, lg);
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int tt = wave; tt < kRouteTok; tt += kRouteThreads / 64) {
    const int t = t0 + tt;
    if (t >= T) break;
    // logits out (fp32, [T][E])
    for (int e = lane; e < E; e += 64) {
      logits_ws[(size_t)t * E + e] = lg[tt][e];
      if (logits_out) logits_out[(size_t)t * E + e] = lg[tt][e];
    }
    // top-k: repeatedly take the largest (value, then lower index) key
    uint32_t khi[MIRA_MAX_EXPERTS / 64], klo[MIRA_MAX_EXPERTS / 64];
#pragma unroll
    for (int i = 0; i < MIRA_MAX_EXPERTS / 64; ++i) {
      const int e = lane + 64 * i;
      khi[i] = e < E ? f32_order_key(lg[tt][e]) : 0u;
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
        my_v = lg[tt][e_sel];
      }
      if (lane == (e_sel & 63)) {
#pragma unroll
        for (int i = 0; i < MIRA_MAX_EXPERTS / 64; ++i)
          if (i == (e_sel >> 6)) khi[i] = klo[i] = 0u;
      }
    }
    // combine weights: softmax over the selected logits (or over all E)
    const float vmax = __shfl(my_v, 0, 64);
    float ex = lane < k ? expf(my_v - vmax) : 0.f;
    float denom;
    if (softmax_all) {
      float s = 0.f;
      for (int e = lane; e < E; e += 64) s += expf(lg[tt][e] - vmax);
      denom = wave_sum(s);
    } else {
      denom = wave_sum(ex);
    }
    if (lane < k) {
      idx_ws[(size_t)t * k + lane] = my_e;
      w_ws[(size_t)t * k + lane] = ex / denom;
    }
  }
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

// ---------------------------------------------------------------------------
// Stable grouping of (token, slot) pairs by expert (one workgroup).
// Routed pair p = t*k + j goes to expert idx[p]; shared expert s owns pairs
// T*k + s*T + t.  Groups: routed experts 0..E-1 then shared 0..S-1; inside a
// group pairs keep increasing p.  Outputs: counts, offsets, inv[p] = position,
// tokpos/wpos (token and combine weight of each position), the list of
// non-empty groups, the prefill m-tile table, and residency status bits.
// The ranks come from wave ballots, never from the order of atomics, so the
// result is deterministic.
// ---------------------------------------------------------------------------
constexpr int kPermThreads = 1024;
constexpr int kPermWaves = kPermThreads / 64;

__global__ __launch_bounds__(kPermThreads) void permute_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ wts, int T, int k, int E, int S,
    int BM, ExpertPool ep, int32_t* __restrict__ counts_ws, int32_t* __restrict__ offsets,
    int32_t* __restrict__ inv, int32_t* __restrict__ tokpos, float* __restrict__ wpos,
    int32_t* __restrict__ misc, int32_t* __restrict__ active, int32_t* __restrict__ mstart,
    int32_t* __restrict__ mtile_g, int32_t* __restrict__ mtile_m0,
    int32_t* __restrict__ counts_out, int32_t* __restrict__ idx_out, float* __restrict__ w_out,
    int32_t* __restrict__ offsets_out, int32_t* __restrict__ order_out) {
  __shared__ int hist[kPermWaves][MIRA_MAX_EXPERTS];
  __shared__ int off_s[MIRA_MAX_EXPERTS + 1];
  __shared__ int mst_s[MIRA_MAX_EXPERTS + 1];
  __shared__ int act_s[MIRA_MAX_EXPERTS];
  __shared__ int n_act_s;
  __shared__ int status_s;
  const int G = E + S, Tk = T * k;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  for (int i = tid; i < kPermWaves * MIRA_MAX_EXPERTS; i += kPermThreads) (&hist[0][0])[i] = 0;
  if (tid == 0) status_s = 0;
  __syncthreads();

  // pass 1: per-wave histograms over contiguous ranges of routed pairs
  const int span = (Tk + kPermWaves - 1) / kPermWaves;
  const int p_beg = wave * span, p_end = min(Tk, p_beg + span);
  for (int p = p_beg + lane; p < p_end; p += 64) {
    const int e = idx[p];
    atomicAdd(&hist[wave][e], 1);
    if (idx_out) idx_out[p] = e;
    if (w_out) w_out[p] = wts[p];
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
        for (int w = 0; w < kPermWaves; ++w) c += hist[w][g];
      } else if (g < G) {
        c = T;
      }
      c4[i] = c;
      sum += c;
    }
    int incl = sum;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const int v = __shfl_up(incl, o, 64);
      if (lane >= o) incl += v;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = lane * 4 + i;
      if (g < G) {
        off_s[g] = run;
        counts_ws[g] = c4[i];
        if (counts_out) counts_out[g] = c4[i];
      }
      run += c4[i];
    }
    if (lane == 63) off_s[G] = incl;  // total pairs
  }
  __syncthreads();
  for (int g = tid; g <= G; g += kPermThreads) {
    offsets[g] = off_s[g];
    if (offsets_out) offsets_out[g] = off_s[g];
  }
  // per-wave bases: offset of the group plus pairs of earlier waves
  for (int g = tid; g < E; g += kPermThreads) {
    int b = off_s[g];
    for (int w = 0; w < kPermWaves; ++w) {
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
    // all lanes read their base before any leader updates it
    __builtin_amdgcn_wave_barrier();
    if (ok) {
      const int pos = b0 + rank;
      inv[p] = pos;
      tokpos[pos] = p / k;
      wpos[pos] = wts[p];
      if (order_out) order_out[pos] = p;
    }
    if (leader) hist[wave][e] = b0 + __popcll(same);
    __builtin_amdgcn_wave_barrier();
  }
  // shared experts: every token, in token order, weight 1
  for (int i = tid; i < S * T; i += kPermThreads) {
    const int s = i / T, t = i - s * T;
    const int pos = off_s[E + s] + t;
    inv[Tk + i] = pos;
    tokpos[pos] = t;
    wpos[pos] = 1.0f;
    if (order_out) order_out[pos] = Tk + i;
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
    for (int o = 1; o < 64; o <<= 1) {
      const int va = __shfl_up(ia, o, 64), vm = __shfl_up(im, o, 64);
      if (lane >= o) {
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
  for (int g = tid; g <= G; g += kPermThreads) mstart[g] = mst_s[g];
  for (int a = tid; a < n_act_s; a += kPermThreads) active[a] = act_s[a];
  for (int g = wave; g < G; g += kPermWaves) {
    const int m0 = mst_s[g], nmt = mst_s[g + 1] - m0;
    for (int m = lane; m < nmt; m += 64) {
      mtile_g[m0 + m] = g;
      mtile_m0[m0 + m] = off_s[g] + m * BM;
    }
  }
  if (tid == 0) {
    misc[MISC_NACTIVE] = n_act_s;
    misc[MISC_MTOTAL] = mst_s[G];
    if (ep.status) *ep.status = status_s;
  }
}

hipError_t launch_permute(const mira_shape& s, const Layout& L, const WsPtr& w,
                          const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                          float* wts_out, int32_t* offsets_out, int32_t* order_out,
                          hipStream_t st) {
  prof_begin("permute", st);
  hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(kPermThreads), 0, st, w.idx, w.wts, L.T, L.k,
                     L.E, L.S, kPrefBM, ep, w.counts, w.offsets, w.inv, w.tokpos, w.wpos, w.misc,
                     w.active, w.mstart, w.mtile_g, w.mtile_m0, counts_out, idx_out, wts_out,
                     offsets_out, order_out);
  prof_end("permute", st);
  return hipGetLastError();
}

__global__ void set_slot_kernel(int32_t* table, int expert, int slot) { table[expert] = slot; }

hipError_t launch_set_slot(int32_t* table, int expert, int slot, hipStream_t st) {
  hipLaunchKernelGGL(set_slot_kernel, dim3(1), dim3(1), 0, st, table, expert, slot);
  return hipGetLastError();
}

}  // namespace mira
