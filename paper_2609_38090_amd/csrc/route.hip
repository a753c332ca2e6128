// Router logits, top-k selection, combine weights and the stable
// token-to-expert permutation (paper section II-A: the router scores every
// expert for each token, the top-k experts process it, their outputs are
// combined).
//
// Two launch shapes share the device functions below:
//  - prefill: route_kernel (16 tokens per workgroup), or with more than 16
//    experts route_tile_kernel (one workgroup per 16 tokens and expert tile)
//    and topk_kernel; then the permutation (one workgroup, or count and
//    scatter kernels over chunks of pairs);
//  - decode (T <= MIRA_DECODE_MAX_TOKENS): one workgroup runs router, top-k,
//    permutation and the fixed-point digits of x back to back, so the
//    expert kernels start after a single small launch.
#include "route_dev.h"

namespace mira {

// Prefill routing, 16 tokens per workgroup: logits with the k range split
// over the 16 waves (the same arithmetic as the decode preparation, so both
// paths route a token identically), then one wave per token for the top-k.
template <typename ActT>
__global__ __launch_bounds__(kBigThreads) void route_kernel(
    const ActT* __restrict__ x, const ActT* __restrict__ wr, const float* __restrict__ bias,
    int T, int E, int C, int k, int softmax_all, int tpw, float* __restrict__ logits_ws,
    float* __restrict__ logits_out, int32_t* __restrict__ idx_ws, float* __restrict__ w_ws) {
  __shared__ float lg[kRouteTok][MIRA_MAX_EXPERTS];
  __shared__ float part[kBigWaves][16][17];
  __shared__ float bias_s[MIRA_MAX_EXPERTS];
  __shared__ int sel_e[kBigWaves][MIRA_MAX_TOPK];
  __shared__ float sel_v[kBigWaves][MIRA_MAX_TOPK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * tpw, nt = min(tpw, T - t0);  // tpw tokens per workgroup
  float bias_r[MIRA_MAX_EXPERTS / kBigThreads + 1];
#pragma unroll
  for (int i = 0; i <= MIRA_MAX_EXPERTS / kBigThreads; ++i) {
    const int e = tid + i * kBigThreads;
    bias_r[i] = (bias && e < E) ? bias[e] : 0.f;
  }
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i <= MIRA_MAX_EXPERTS / kBigThreads; ++i) {
      const int e = tid + i * kBigThreads;
      if (e < E) bias_s[e] = bias_r[i];
    }
  };
  if constexpr (sizeof(ActT) == 2) {
    logits_ksplit_bf16(x + (size_t)t0 * C, wr, bias_s, nt, E, C, part, lg, nullptr, stage);
  } else {
    logits_tile_f32(x, wr, bias, T, E, C, t0, kBigWaves, lg);
    __syncthreads();
  }
  if (wave < nt) {
    const int t = t0 + wave;
    for (int e = lane; e < E; e += 64) {
      logits_ws[(size_t)t * E + e] = lg[wave][e];
      if (logits_out) logits_out[(size_t)t * E + e] = lg[wave][e];
    }
    topk_rank(lg[wave], E, k, softmax_all, idx_ws + (size_t)t * k, w_ws + (size_t)t * k,
              sel_e[wave], sel_v[wave]);
  }
}


// Prefill routing over several expert tiles (bf16, E > 16): one workgroup
// per (16 tokens, tile of 16 experts), each tile summed exactly as above,
// logits to the workspace; topk_kernel then selects.  So the tiles of a
// token group run side by side on different CUs.
__global__ __launch_bounds__(kBigThreads) void route_tile_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wr, const float* __restrict__ bias,
    int T, int E, int C, int tpw, float* __restrict__ logits_ws, float* __restrict__ logits_out) {
  __shared__ float lg[kRouteTok][MIRA_MAX_EXPERTS];
  __shared__ float part[kBigWaves][16][17];
  __shared__ float bias_s[MIRA_MAX_EXPERTS];
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * tpw, nt = min(tpw, T - t0), et = blockIdx.y;
  const int e_lo = et * 16, ne = min(16, E - e_lo);
  const float b_r = (bias && tid < ne) ? bias[e_lo + tid] : 0.f;
  auto stage = [&]() {
    if (tid < ne) bias_s[e_lo + tid] = b_r;
  };
  logits_ksplit_bf16(x + (size_t)t0 * C, wr, bias ? bias_s : nullptr, nt, E, C, part, lg, nullptr,
                     stage, et, et + 1);
  if (tid < nt * 16) {
    const int tt = tid >> 4, ee = tid & 15;
    if (ee < ne) {
      const size_t i = (size_t)(t0 + tt) * E + e_lo + ee;
      logits_ws[i] = lg[tt][e_lo + ee];
      if (logits_out) logits_out[i] = lg[tt][e_lo + ee];
    }
  }
}

// Top-k and combine weights from the workspace logits, one wave per token.
__global__ __launch_bounds__(kBigThreads) void topk_kernel(const float* __restrict__ logits_ws,
                                                           int T, int E, int k, int softmax_all,
                                                           int32_t* __restrict__ idx_ws,
                                                           float* __restrict__ w_ws) {
  __shared__ int sel_e[kBigWaves][MIRA_MAX_TOPK];
  __shared__ float sel_v[kBigWaves][MIRA_MAX_TOPK];
  const int wave = threadIdx.x >> 6;
  const int t = blockIdx.x * kBigWaves + wave;
  if (t >= T) return;
  topk_rank(logits_ws + (size_t)t * E, E, k, softmax_all, idx_ws + (size_t)t * k,
            w_ws + (size_t)t * k, sel_e[wave], sel_v[wave]);
}

// Group counts and their exclusive scan (wave 0; each lane owns 4
// consecutive groups): routed group g < E holds count(g) pairs, shared group
// E + s holds T.  Writes off_s[0..G] in LDS and the counts outputs.
template <typename CountFn>
__device__ void group_offsets(CountFn count, int T, int E, int S, int* off_s, const PermOut& o) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, G = E + S;
  if (wave != 0) return;
  int c4[4], sum = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int g = lane * 4 + i;
    const int c = g < E ? count(g) : (g < G ? T : 0);
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

// Group tables shared by both permutation shapes, from the group offsets
// off_s[0..G] in LDS: the list of non-empty groups, residency status bits,
// and the prefill m-tile prefix (tiles of BM positions).  Called by every
// thread of one workgroup.
__device__ void group_tables(const int* off_s, int G, int BM, const ExpertPool& ep,
                             const PermOut& o) {
  __shared__ int mst_s[MIRA_MAX_EXPERTS + 1];
  __shared__ int act_s[MIRA_MAX_EXPERTS];
  __shared__ int n_act_s;
  __shared__ int status_s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) status_s = 0;
  __syncthreads();
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

__device__ void permute_body(const int32_t* idx, const float* wts, int T, int k, int E, int S,
                             int BM, const ExpertPool& ep, const PermOut& o) {
  __shared__ int hist[kBigWaves][MIRA_MAX_EXPERTS];
  __shared__ int off_s[MIRA_MAX_EXPERTS + 1];
  const int G = E + S, Tk = T * k;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

  for (int i = tid; i < kBigWaves * MIRA_MAX_EXPERTS; i += kBigThreads) (&hist[0][0])[i] = 0;
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

  // counts and exclusive scan
  group_offsets([&](int g) {
    int c = 0;
    for (int w = 0; w < kBigWaves; ++w) c += hist[w][g];
    return c;
  }, T, E, S, off_s, o);
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

  group_tables(off_s, G, BM, ep, o);
}

// Chunked permutation, first pass: counts of each expert among the routed
// pairs of chunk blockIdx.x (pcnt[chunk][e]); also copies idx/wts out.
__global__ __launch_bounds__(kBigThreads) void permute_count_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ wts, int Tk, int E,
    int32_t* __restrict__ pcnt, int32_t* __restrict__ idx_out, float* __restrict__ w_out) {
  __shared__ int h[MIRA_MAX_EXPERTS];
  const int tid = threadIdx.x;
  for (int e = tid; e < E; e += kBigThreads) h[e] = 0;
  __syncthreads();
  const int p = blockIdx.x * kPermChunk + tid;
  if (p < Tk) {
    const int e = idx[p];
    atomicAdd(&h[e], 1);
    if (idx_out) idx_out[p] = e;
    if (w_out) w_out[p] = wts[p];
  }
  __syncthreads();
  for (int e = tid; e < E; e += kBigThreads) pcnt[blockIdx.x * E + e] = h[e];
}

// Chunked permutation, second pass (one workgroup per chunk, one thread per
// pair): the position of a pair is the group offset, plus the pairs of the
// same expert in earlier chunks, earlier waves of this chunk and earlier
// lanes of its wave (ballot ranks), so the result equals the one-workgroup
// permutation.  Each workgroup also places a share of the shared-expert
// pairs; workgroup 0 writes the group tables.
__global__ __launch_bounds__(kBigThreads) void permute_scatter_kernel(
    const int32_t* __restrict__ idx, const float* __restrict__ wts, int T, int k, int E, int S,
    int BM, int nchunk, const int32_t* __restrict__ pcnt, ExpertPool ep, PermOut o) {
  __shared__ int hist[kBigWaves][MIRA_MAX_EXPERTS];
  __shared__ int tot_s[MIRA_MAX_EXPERTS], pre_s[MIRA_MAX_EXPERTS];
  __shared__ int off_s[MIRA_MAX_EXPERTS + 1];
  const int G = E + S, Tk = T * k, c = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  for (int e = tid; e < E; e += kBigThreads) {
    int tot = 0, pre = 0;
    for (int cc = 0; cc < nchunk; ++cc) {
      const int v = pcnt[cc * E + e];
      tot += v;
      pre += cc < c ? v : 0;
    }
    tot_s[e] = tot;
    pre_s[e] = pre;
  }
  // this thread's pair and its rank among the same expert's pairs of the wave
  const int p = c * kPermChunk + tid;
  const bool ok = p < Tk;
  const int e = ok ? idx[p] : 0;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  uint64_t same = __ballot(ok);
#pragma unroll
  for (int bit = 0; bit < 8; ++bit) {
    const uint64_t b = __ballot(ok && ((e >> bit) & 1));
    same &= ((e >> bit) & 1) ? b : ~b;
  }
  const int rank = __popcll(same & lt_mask);
  for (int i = tid; i < kBigWaves * MIRA_MAX_EXPERTS; i += kBigThreads) (&hist[0][0])[i] = 0;
  __syncthreads();
  if (ok && (same & lt_mask) == 0) hist[wave][e] = __popcll(same);  // one leader per expert
  group_offsets([&](int g) { return tot_s[g]; }, T, E, S, off_s, o);
  __syncthreads();
  // bases of each wave: group offset + earlier chunks + earlier waves
  for (int g = tid; g < E; g += kBigThreads) {
    int b = off_s[g] + pre_s[g];
    for (int w = 0; w < kBigWaves; ++w) {
      const int n = hist[w][g];
      hist[w][g] = b;
      b += n;
    }
  }
  __syncthreads();
  if (ok) {
    const int pos = hist[wave][e] + rank;
    o.inv[p] = pos;
    o.tokpos[pos] = p / k;
    o.wpos[pos] = wts[p];
    if (o.order_out) o.order_out[pos] = p;
  }
  // shared experts: every token, in token order, weight 1
  const int span = (S * T + nchunk - 1) / nchunk;
  for (int i = c * span + tid; i < min(S * T, (c + 1) * span); i += kBigThreads) {
    const int s = i / T, t = i - s * T;
    const int pos = off_s[E + s] + t;
    o.inv[Tk + i] = pos;
    o.tokpos[pos] = t;
    o.wpos[pos] = 1.0f;
    if (o.order_out) o.order_out[pos] = Tk + i;
  }
  if (c == 0) {
    for (int g = tid; g <= G; g += kBigThreads) {
      o.offsets[g] = off_s[g];
      if (o.offsets_out) o.offsets_out[g] = off_s[g];
    }
    group_tables(off_s, G, BM, ep, o);
  }
}

__global__ __launch_bounds__(kBigThreads) void permute_kernel(const int32_t* __restrict__ idx,
                                                              const float* __restrict__ wts, int T,
                                                              int k, int E, int S, int BM,
                                                              ExpertPool ep, PermOut o) {
  permute_body(idx, wts, T, k, E, S, BM, ep, o);
}


// ---------------------------------------------------------------------------
// Decode preparation (T <= 16 tokens, one workgroup): router logits (with
// max |x| per token on the way), top-k and weights; then wave 0 groups the
// pairs (with wave 1 writing the optional outputs when there are at most 64
// pairs) while the other waves write the fixed-point digits of x used by the
// integer expert kernels (|x * 2^E_t| < 2^22 per token, three signed
// base-256 digits; layout xdig[(t*3 + d)*C + c]; the exponent E_t goes into
// the expert descriptors).
// ---------------------------------------------------------------------------
// Fixed-point digits (exponent Ex) of elements 4*i .. 4*i+3 of one token's x
// row xr, into that token's three digit rows xd[d*C + c].
template <typename ActT>
__device__ __forceinline__ void write_x_digits4(const ActT* __restrict__ xr, int i, int Ex,
                                                int8_t* __restrict__ xd, int C) {
  const int c = i * 4;
  float v[4];
  load4_act(xr + c, v);
  uint32_t w0 = 0, w1 = 0, w2 = 0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    int d0, d1, d2;
    split_digits((int)rintf(ldexpf(v[j], Ex)), d0, d1, d2);
    w0 |= (uint32_t)(d0 & 0xFF) << (8 * j);
    w1 |= (uint32_t)(d1 & 0xFF) << (8 * j);
    w2 |= (uint32_t)(d2 & 0xFF) << (8 * j);
  }
  *(uint32_t*)(xd + c) = w0;
  *(uint32_t*)(xd + C + c) = w1;
  *(uint32_t*)(xd + 2 * (size_t)C + c) = w2;
}

template <typename ActT>
__global__ __launch_bounds__(kBigThreads) void decode_prep_kernel(
    const ActT* __restrict__ x, const ActT* __restrict__ wr, const float* __restrict__ bias,
    int T, int E, int C, int k, int S, int softmax_all, float* __restrict__ logits_out,
    ExpertPool ep, PermOut o, DecodeWork* __restrict__ work, int max_active,
    int8_t* __restrict__ xdig) {
  __shared__ float lg[kRouteTok][MIRA_MAX_EXPERTS];
  __shared__ float part[kBigWaves][16][17];
  __shared__ int32_t idx_s[kRouteTok * MIRA_MAX_TOPK];
  __shared__ float w_s[kRouteTok * MIRA_MAX_TOPK];
  __shared__ float xmax[kRouteTok];
  __shared__ int xe_s[kRouteTok];
  __shared__ int cnt_s[MIRA_MAX_EXPERTS], run_s[MIRA_MAX_EXPERTS];
  __shared__ int ptok_s[kDecodeMaxPairs];
  __shared__ float pw_s[kDecodeMaxPairs];
  __shared__ float bias_s[MIRA_MAX_EXPERTS];
  __shared__ int slot_s[MIRA_MAX_EXPERTS];
  __shared__ int sel_e[kRouteTok][MIRA_MAX_TOPK];
  __shared__ float sel_v[kRouteTok][MIRA_MAX_TOPK];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // load the router bias and the slot table into registers now and store
  // them to LDS just before the logits barrier, so the loads overlap
  float bias_r[MIRA_MAX_EXPERTS / kBigThreads + 1];
  int slot_r[MIRA_MAX_EXPERTS / kBigThreads + 1];
#pragma unroll
  for (int i = 0; i <= MIRA_MAX_EXPERTS / kBigThreads; ++i) {
    const int e = tid + i * kBigThreads;
    bias_r[i] = (bias && e < E) ? bias[e] : 0.f;
    slot_r[i] = e < E + S ? ep.slot_table[e] : 0;
  }
  auto stage = [&]() {
#pragma unroll
    for (int i = 0; i <= MIRA_MAX_EXPERTS / kBigThreads; ++i) {
      const int e = tid + i * kBigThreads;
      if (e < E) bias_s[e] = bias_r[i];
      if (e < E + S) slot_s[e] = slot_r[i];
    }
  };

  if constexpr (sizeof(ActT) == 2) {
    logits_ksplit_bf16(x, wr, bias_s, T, E, C, part, lg, xmax, stage);
  } else {
    stage();
    logits_tile_f32(x, wr, bias, T, E, C, 0, kBigWaves, lg);
    if (wave < T) {  // one wave per token: max |x|
      float m = 0.f;
      for (int c = lane * 4; c < C; c += 256) {
        float v[4];
        load4_act(x + (size_t)wave * C + c, v);
        m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
      }
      m = wave_max(m);
      if (lane == 0) xmax[wave] = m;
    }
    __syncthreads();
  }
  if (T == 1 && E <= 64 && k + S <= 64) {
    // one token: nothing waits after the logits.  Wave 0 selects and writes
    // the descriptors from registers; wave 1 makes the same selection (same
    // keys, same order) for the optional outputs; the other waves write the
    // digits of x.
    const int xe = kFixBits - exp_bound(xmax[0]);
    if (wave == 0) {
      decode_work_one_token(lg[0], E, k, S, softmax_all, xe, slot_s, ep, work, max_active);
    } else if (wave == 1) {
      if (logits_out)
        for (int e = lane; e < E; e += 64) logits_out[e] = lg[0][e];
      topk_rank(lg[0], E, k, softmax_all, idx_s, w_s, sel_e[0], sel_v[0]);
      decode_outputs_small(idx_s, w_s, 1, k, E, S, o, cnt_s);
    } else {
      for (int i = tid - 128; i < C / 4; i += kBigThreads - 128) write_x_digits4(x, i, xe, xdig, C);
    }
    return;
  }
  if (wave < T) {
    const int t = wave;
    if (logits_out)
      for (int e = lane; e < E; e += 64) logits_out[(size_t)t * E + e] = lg[t][e];
    topk_rank(lg[t], E, k, softmax_all, idx_s + t * k, w_s + t * k, sel_e[t], sel_v[t]);
  }
  if (tid < T) xe_s[tid] = kFixBits - exp_bound(xmax[tid]);
  lds_barrier();  // the routing and exponents are in LDS; no global data is read after this

  // up to 64 pairs: wave 0 writes the expert kernels' descriptors and wave 1
  // the optional outputs side by side; otherwise wave 0 does both
  const bool small = T * k <= kDecodeSmallPairs;
  if (wave == 0) {
    if (small)
      decode_work_small(idx_s, w_s, xe_s, slot_s, T, k, E, S, ep, work, max_active);
    else
      permute_decode_wave(idx_s, w_s, xe_s, slot_s, T, k, E, S, ep, o, work, max_active, cnt_s,
                          run_s, ptok_s, pw_s);
    return;
  }
  if (small && wave == 1) {
    decode_outputs_small(idx_s, w_s, T, k, E, S, o, cnt_s);
    return;
  }
  // the other waves: fixed-point digits of x, four elements per thread and step
  const int w0d = small ? 2 : 1;
  const int q4 = C / 4, n4 = T * q4;
  for (int i = tid - 64 * w0d; i < n4; i += kBigThreads - 64 * w0d) {
    const int t = i / q4;
    write_x_digits4(x + (size_t)t * C, i - t * q4, xe_s[t], xdig + (size_t)t * kDigits * C, C);
  }
}


hipError_t launch_route(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                        const void* wr, const float* bias, float* logits_out, hipStream_t st) {
  const int T = L.T;
  if (T == 0) return hipSuccess;
  // bf16 with one expert tile: a few tokens per workgroup, so the 16 router
  // rows (read by every workgroup) stream into many CUs at once; a token's
  // sums do not depend on which other tokens share its MFMA operand.  With
  // several tiles, more workgroups would re-read every tile's rows.
  const int n_et = (L.E + 15) / 16;
  const int tpw = (s.act_dtype == MIRA_BF16 && n_et == 1) ? kRouteTokBf16 : kRouteTok;
  dim3 grid((T + tpw - 1) / tpw), block(kBigThreads);
  const int sa = (s.flags & MIRA_FLAG_SOFTMAX_ALL) ? 1 : 0;
  prof_begin("route", st);
  if (s.act_dtype == MIRA_BF16 && n_et > 1) {
    hipLaunchKernelGGL(route_tile_kernel, dim3(grid.x, n_et), block, 0, st, (const uint16_t*)x,
                       (const uint16_t*)wr, bias, T, L.E, L.C, tpw, w.logits, logits_out);
    hipLaunchKernelGGL(topk_kernel, dim3((T + kBigWaves - 1) / kBigWaves), block, 0, st,
                       (const float*)w.logits, T, L.E, L.k, sa, w.idx, w.wts);
  } else if (s.act_dtype == MIRA_BF16)
    hipLaunchKernelGGL(route_kernel<uint16_t>, grid, block, 0, st, (const uint16_t*)x,
                       (const uint16_t*)wr, bias, T, L.E, L.C, L.k, sa, tpw, w.logits, logits_out,
                       w.idx, w.wts);
  else
    hipLaunchKernelGGL(route_kernel<float>, grid, block, 0, st, (const float*)x,
                       (const float*)wr, bias, T, L.E, L.C, L.k, sa, tpw, w.logits, logits_out,
                       w.idx, w.wts);
  prof_end("route", st);
  return hipGetLastError();
}

hipError_t launch_permute(const Layout& L, const WsPtr& w,
                          const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                          float* wts_out, int32_t* offsets_out, int32_t* order_out,
                          hipStream_t st) {
  const PermOut o = perm_out(w, counts_out, idx_out, wts_out, offsets_out, order_out);
  const int Tk = L.T * L.k, nchunk = (Tk + kPermChunk - 1) / kPermChunk;
  prof_begin("permute", st);
  if (nchunk >= 2 && nchunk <= kPermChunkMax) {
    hipLaunchKernelGGL(permute_count_kernel, dim3(nchunk), dim3(kBigThreads), 0, st, w.idx, w.wts,
                       Tk, L.E, w.pcnt, idx_out, wts_out);
    hipLaunchKernelGGL(permute_scatter_kernel, dim3(nchunk), dim3(kBigThreads), 0, st, w.idx,
                       w.wts, L.T, L.k, L.E, L.S, kPrefBM, nchunk, (const int32_t*)w.pcnt, ep, o);
  } else {
    hipLaunchKernelGGL(permute_kernel, dim3(1), dim3(kBigThreads), 0, st, w.idx, w.wts, L.T, L.k,
                       L.E, L.S, kPrefBM, ep, o);
  }
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
  const int max_active = decode_max_active(L);
  prof_begin("decode_prep", st);
  if (s.act_dtype == MIRA_BF16)
    hipLaunchKernelGGL(decode_prep_kernel<uint16_t>, dim3(1), dim3(kBigThreads), 0, st,
                       (const uint16_t*)x, (const uint16_t*)wr, bias, L.T, L.E, L.C, L.k, L.S, sa,
                       logits_out, ep, o, w.dwork, max_active, w.xdig);
  else
    hipLaunchKernelGGL(decode_prep_kernel<float>, dim3(1), dim3(kBigThreads), 0, st,
                       (const float*)x, (const float*)wr, bias, L.T, L.E, L.C, L.k, L.S, sa,
                       logits_out, ep, o, w.dwork, max_active, w.xdig);
  prof_end("decode_prep", st);
  return hipGetLastError();
}

// A whole slot-table row, passed by value (at most MIRA_MAX_EXPERTS entries).
struct TableRow {
  int32_t v[MIRA_MAX_EXPERTS];
};

__global__ void set_table_kernel(int32_t* table, TableRow row, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) table[i] = row.v[i];
}

hipError_t launch_set_table(int32_t* table, const int32_t* row, int n, hipStream_t st) {
  if (n < 1 || n > MIRA_MAX_EXPERTS) return hipErrorInvalidValue;
  TableRow r;
  for (int i = 0; i < n; ++i) r.v[i] = row[i];
  hipLaunchKernelGGL(set_table_kernel, dim3(1), dim3(256), 0, st, table, r, n);
  return hipGetLastError();
}

__global__ void set_slot_kernel(int32_t* table, int expert, int slot) { table[expert] = slot; }

hipError_t launch_set_slot(int32_t* table, int expert, int slot, hipStream_t st) {
  hipLaunchKernelGGL(set_slot_kernel, dim3(1), dim3(1), 0, st, table, expert, slot);
  return hipGetLastError();
}

}  // namespace mira
