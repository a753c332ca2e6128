// Device-side routing helpers of the routing kernels: router logits for up
// to 16 tokens, top-k by rank counting with the combine weights, and the
// one-wave stable grouping of a decode call's (token, slot) pairs (paper section II-A: the router scores every
// expert, the top-k experts process the token, their outputs are combined).
#pragma once

#include "device_util.h"
#include "mira_internal.h"

namespace mira {

constexpr int kRouteTok = 16;  // tokens per route workgroup (at most)
constexpr int kRouteTokBf16 = 4;  // tokens per prefill route workgroup, bf16, one expert tile
constexpr int kBigThreads = 1024;  // permutation and decode-prep workgroups
static_assert(kPermChunk == kBigThreads, "the chunked permutation runs one thread per pair");
constexpr int kBigWaves = kBigThreads / 64;

// ---------------------------------------------------------------------------
// Router logits for 16 tokens: lg[t][e] = sum_c x[t][c] * Wg[e][c] + b[e].
// fp32: VALU dot products, one wave per (token, expert), fp32 accumulate.
// bf16 (below): MFMA, A = Wg rows (experts), B = x rows (tokens), fp32
// accumulate, the k range split over the waves.
// ---------------------------------------------------------------------------
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

// Workgroup barrier for LDS traffic only: global loads still in flight (the
// next expert tile's router rows) are not drained, unlike __syncthreads.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// bf16 logits for up to 16 tokens (decode preparation and prefill routing
// alike): all waves of the workgroup split the k range of every expert tile;
// partial sums are reduced through LDS in wave order.
__device__ __forceinline__ float absmax_bf16x8(v4i v) {
  float m = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t u = (uint32_t)v[i];
    m = fmaxf(m, fmaxf(fabsf(__uint_as_float(u << 16)), fabsf(__uint_as_float(u & 0xFFFF0000u))));
  }
  return m;
}

// x points at the first of T <= 16 tokens.  If xmax is not null it also
// receives max |x[t][:]| of each token; bias_s is the router bias (or null),
// staged into LDS by pre_sync() right before the first barrier.  Expert
// tiles et_begin .. et_end-1 of 16 experts are computed (all by default);
// a tile's sums do not depend on which other tiles the call computes.
template <typename PreSync>
__device__ void logits_ksplit_bf16(const uint16_t* __restrict__ x, const uint16_t* __restrict__ wr,
                                   const float* bias_s, int T, int E, int C,
                                   float (*part)[16][17], float (*lg)[MIRA_MAX_EXPERTS],
                                   float* xmax, PreSync pre_sync, int et_begin = 0,
                                   int et_end = -1) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int n_et = et_end < 0 ? (E + 15) / 16 : et_end, nch = C / 32;
  const bool tok_ok = r16 < T;
  const uint16_t* xrow = x + (size_t)(tok_ok ? r16 : 0) * C + kg * 8;
  constexpr int B = 8;  // chunks in flight per wave
  // When one batch of chunks covers the k range (C <= 4096) the next expert
  // tile's router rows are loaded while the current tile is reduced.
  const bool one_batch = nch <= B * kBigWaves;
  v4i a[B];
  auto load_rows = [&](int et) {
    const int e = et * 16 + r16;
    const bool e_ok = e < E;
    const uint16_t* wrow = wr + (size_t)(e_ok ? e : 0) * C + kg * 8;
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const int ch = wave + u * kBigWaves;
      a[u] = (ch < nch && e_ok) ? ld16(wrow + ch * 32) : zero16();
    }
  };
  if (one_batch) load_rows(et_begin);
  for (int et = et_begin; et < n_et; ++et) {
    v4f acc = {0.f, 0.f, 0.f, 0.f};
    float xm = 0.f;
    for (int ch0 = wave; ch0 < nch; ch0 += B * kBigWaves) {
      if (!one_batch) {
        const int e = et * 16 + r16;
        const bool e_ok = e < E;
        const uint16_t* wrow = wr + (size_t)(e_ok ? e : 0) * C + kg * 8;
#pragma unroll
        for (int u = 0; u < B; ++u) {
          const int ch = ch0 + u * kBigWaves;
          a[u] = (ch < nch && e_ok) ? ld16(wrow + ch * 32) : zero16();
        }
      }
      v4i b[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int ch = ch0 + u * kBigWaves;
        b[u] = (ch < nch && tok_ok) ? ld16(xrow + ch * 32) : zero16();
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        acc = mfma_bf16(a[u], b[u], acc);
        if (et == et_begin) xm = fmaxf(xm, absmax_bf16x8(b[u]));
      }
    }
    if (one_batch && et + 1 < n_et) load_rows(et + 1);
#pragma unroll
    for (int i = 0; i < 4; ++i) part[wave][r16][kg * 4 + i] = acc[i];  // [token][expert]
    if (et == et_begin) {
      // this wave's max over its chunks of token r16: combine the 4 lane groups
      xm = fmaxf(xm, __shfl_xor(xm, 16, 64));
      xm = fmaxf(xm, __shfl_xor(xm, 32, 64));
      if (kg == 0) part[wave][r16][16] = xm;  // column 16 is spare
      pre_sync();  // caller's LDS staging, issued before the loads above
    }
    lds_barrier();
    if (et == et_begin && xmax && tid < 16) {
      float m = 0.f;
      for (int w = 0; w < kBigWaves; ++w) m = fmaxf(m, part[w][tid][16]);
      xmax[tid] = m;
    }
    if (tid < 256) {
      const int tt = tid >> 4, ee = tid & 15, e2 = et * 16 + ee;
      float s = 0.f;
      for (int w = 0; w < kBigWaves; ++w) s += part[w][tt][ee];
      if (e2 < E) lg[tt][e2] = s + (bias_s ? bias_s[e2] : 0.f);
    }
    lds_barrier();
  }
}

// Top-k of one token by rank counting (one wave): expert e is selected at
// position rank(e) = number of experts with a larger (value, then lower
// index) key, if that is < k.  Each lane holds the logits of its experts
// (lane, lane+64, ...) in registers and takes every other expert's key with
// v_readlane, so the count needs no memory round trips.  The combine weights
// are a softmax in fp32, summed in selection order.  sel_e/sel_v: this wave's
// LDS scratch.
// The selection of topk_rank with E <= 64 experts, one per lane: lane e
// learns whether it is selected, its position and its combine weight.
__device__ __forceinline__ void topk_lane64(const float* lgrow, int E, int k, int softmax_all,
                                            bool& sel, int& rank, float& w) {
  const int lane = threadIdx.x & 63;
  const bool in = lane < E;
  const float v = in ? lgrow[lane] : 0.f;
  const uint32_t key = f32_order_key(v);
  rank = 0;
#pragma unroll 1
  for (int l2 = 0; l2 < E; ++l2) {
    const uint32_t k2 = (uint32_t)__builtin_amdgcn_readlane((int)key, l2);
    rank += (k2 > key) || (k2 == key && l2 < lane);
  }
  sel = in && rank < k;
  const int l0 = __builtin_ctzll(__ballot(sel && rank == 0));
  const float vmax = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l0));
  const float ex = in ? expf(v - vmax) : 0.f;
  float denom = 0.f;
  if (softmax_all) {
    denom = wave_sum(ex);
  } else {
#pragma unroll 1
    for (int j = 0; j < k; ++j) {
      const int lj = __builtin_ctzll(__ballot(sel && rank == j));
      denom += __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ex), lj));
    }
  }
  w = ex / denom;
}

__device__ __forceinline__ void topk_rank(const float* lgrow, int E, int k, int softmax_all,
                                          int32_t* idx_a, float* w_a, int* sel_e, float* sel_v) {
  constexpr int kPer = MIRA_MAX_EXPERTS / 64;  // experts per lane
  const int lane = threadIdx.x & 63;
  if (E <= 64) {
    // one expert per lane: the selection stays in registers (the same keys,
    // exponentials and sum order as below, so the results are identical)
    bool sel;
    int rank;
    float w;
    topk_lane64(lgrow, E, k, softmax_all, sel, rank, w);
    if (sel) {
      idx_a[rank] = lane;
      w_a[rank] = w;
    }
    return;
  }
  const int nblk = (E + 63) / 64;
  // each lane keeps the logits of experts lane, lane+64, ... in registers;
  // the comparison keys of the other experts come from v_readlane
  float val[kPer];
  uint32_t key[kPer];
  int rank[kPer];
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = lane + 64 * i;
    val[i] = e < E ? lgrow[e] : 0.f;
    key[i] = f32_order_key(val[i]);
    rank[i] = 0;
  }
#pragma unroll
  for (int i2 = 0; i2 < kPer; ++i2) {
    if (i2 >= nblk) break;
    const int n2 = min(64, E - 64 * i2);
#pragma unroll 1
    for (int l2 = 0; l2 < n2; ++l2) {
      const uint32_t k2 = (uint32_t)__builtin_amdgcn_readlane((int)key[i2], l2);
      const int e2 = 64 * i2 + l2;
#pragma unroll
      for (int i = 0; i < kPer; ++i)
        if (i < nblk) rank[i] += (k2 > key[i]) || (k2 == key[i] && e2 < lane + 64 * i);
    }
  }
#pragma unroll
  for (int i = 0; i < kPer; ++i) {
    const int e = lane + 64 * i;
    if (e < E && rank[i] < k) {
      sel_e[rank[i]] = e;
      sel_v[rank[i]] = val[i];
    }
  }
  __builtin_amdgcn_wave_barrier();
  const float vmax = sel_v[0];
  float denom = 0.f;
  if (softmax_all) {
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kPer; ++i)
      if (lane + 64 * i < E) s += expf(val[i] - vmax);
    denom = wave_sum(s);
  } else {
#pragma unroll 1
    for (int j = 0; j < k; ++j) denom += expf(sel_v[j] - vmax);
  }
  if (lane < k) {
    idx_a[lane] = sel_e[lane];
    w_a[lane] = expf(sel_v[lane] - vmax) / denom;
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

// ---------------------------------------------------------------------------
// Stable grouping for a decode call (T <= 16 tokens, at most kDecodeMaxPairs
// pairs) by one wave: chunks of 64 pairs in order, ranks from ballots, running
// group bases in LDS.  Same outputs as permute_body, plus one DecodeWork
// descriptor per non-empty group.
// ---------------------------------------------------------------------------
__device__ inline void permute_decode_wave(const int32_t* idx, const float* wts, const int* xe_s,
                                           const int* slot_s, int T, int k, int E, int S,
                                           const ExpertPool& ep, const PermOut& o,
                                           DecodeWork* __restrict__ work, int max_active,
                                           int* cnt_s, int* run_s, int* ptok_s, float* pw_s) {
  // reused once the counts and running bases are consumed: per non-empty group
  int* act_off_s = cnt_s;
  int* act_n_s = run_s;
  const int lane = threadIdx.x & 63;
  const int G = E + S, Tk = T * k;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int g = lane; g < G; g += 64) cnt_s[g] = g >= E ? T : 0;
  __builtin_amdgcn_wave_barrier();
  auto match = [&](bool ok, int e) {
    uint64_t same = __ballot(ok);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const uint64_t bb = __ballot(ok && ((e >> bit) & 1));
      same &= ((e >> bit) & 1) ? bb : ~bb;
    }
    return same;
  };
  for (int base = 0; base < Tk; base += 64) {
    const int p = base + lane;
    const bool ok = p < Tk;
    const int e = ok ? idx[p] : 0;
    const uint64_t same = match(ok, e);
    if (ok && (same & lt_mask) == 0) cnt_s[e] += __popcll(same);
    __builtin_amdgcn_wave_barrier();
    if (ok) {
      if (o.idx_out) o.idx_out[p] = e;
      if (o.w_out) o.w_out[p] = wts[p];
    }
  }
  // one exclusive scan over groups (4 consecutive groups per lane) carrying
  // both the pair count (low 16 bits) and the non-empty group count (high)
  int c4[4], sum = 0, nz = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int g = lane * 4 + i;
    c4[i] = g < G ? cnt_s[g] : 0;
    sum += c4[i];
    nz += c4[i] > 0;
  }
  int packed = sum | (nz << 16);
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(packed, off, 64);
    if (lane >= off) packed += v;
  }
  const int incl = packed & 0xFFFF, ia = packed >> 16, na = nz;
  int run = incl - sum;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int g = lane * 4 + i;
    if (g < G) {
      run_s[g] = run;
      o.counts_ws[g] = c4[i];
      o.offsets[g] = run;
      if (o.counts_out) o.counts_out[g] = c4[i];
      if (o.offsets_out) o.offsets_out[g] = run;
    }
    run += c4[i];
  }
  if (lane == 63) {
    o.offsets[G] = incl;
    if (o.offsets_out) o.offsets_out[G] = incl;
  }
  __builtin_amdgcn_wave_barrier();
  // positions of routed pairs
  for (int base = 0; base < Tk; base += 64) {
    const int p = base + lane;
    const bool ok = p < Tk;
    const int e = ok ? idx[p] : 0;
    const uint64_t same = match(ok, e);
    int b0 = 0;
    if (ok) b0 = run_s[e];
    __builtin_amdgcn_wave_barrier();  // every lane has read its base
    if (ok) {
      const int pos = b0 + __popcll(same & lt_mask);
      const float w = wts[p];
      o.inv[p] = pos;
      o.tokpos[pos] = p / k;
      o.wpos[pos] = w;
      ptok_s[pos] = p / k;
      pw_s[pos] = w;
      if (o.order_out) o.order_out[pos] = p;
      if ((same & lt_mask) == 0) run_s[e] = b0 + __popcll(same);
    }
    __builtin_amdgcn_wave_barrier();
  }
  // shared experts: every token in order, weight 1 (their bases were not advanced)
  for (int i = lane; i < S * T; i += 64) {
    const int s = i / T, t = i - s * T;
    const int pos = run_s[E + s] + t;
    o.inv[Tk + i] = pos;
    o.tokpos[pos] = t;
    o.wpos[pos] = 1.0f;
    ptok_s[pos] = t;
    pw_s[pos] = 1.0f;
    if (o.order_out) o.order_out[pos] = Tk + i;
  }
  __builtin_amdgcn_wave_barrier();
  // non-empty groups in order -> descriptors (headers by the owning lane,
  // then the per-position fields spread over all lanes)
  const int n_active = __shfl(ia, 63, 64);
  int ra = ia - na, bits = 0;
  int gbase = incl - sum;
  for (int i = 0; i < 4; ++i) {
    const int g = lane * 4 + i;
    if (g < G && c4[i] > 0) {
      const int slot = slot_s[g];
      if (slot < 0) bits |= 1;
      else if (slot >= ep.n_slots) bits |= 2;
      o.active[ra] = g;
      DecodeWork* wk = work + ra;
      wk->group = g;
      wk->slot = slot;
      wk->off = gbase;
      wk->n = c4[i];
      act_off_s[ra] = gbase;
      act_n_s[ra] = c4[i];
      ++ra;
    }
    gbase += c4[i];
  }
  __builtin_amdgcn_wave_barrier();
  for (int it = lane; it < n_active * MIRA_DECODE_MAX_TOKENS; it += 64) {
    const int a = it / MIRA_DECODE_MAX_TOKENS, j = it - a * MIRA_DECODE_MAX_TOKENS;
    const int off = act_off_s[a];
    const bool v = j < act_n_s[a];
    const int t = v ? ptok_s[off + j] : 0;
    work[a].tok[j] = t;
    work[a].xe[j] = v ? xe_s[t] : 0;
    work[a].w[j] = v ? pw_s[off + j] : 0.f;
  }
  for (int a = n_active + lane; a < max_active; a += 64) work[a].group = -1;
  bits |= __shfl_xor(bits, 1, 64);
  bits |= __shfl_xor(bits, 2, 64);
  bits |= __shfl_xor(bits, 4, 64);
  bits |= __shfl_xor(bits, 8, 64);
  bits |= __shfl_xor(bits, 16, 64);
  bits |= __shfl_xor(bits, 32, 64);
  if (lane == 0) {
    o.misc[MISC_NACTIVE] = n_active;
    o.misc[MISC_MTOTAL] = 0;
    if (ep.status) *ep.status = bits;
  }
}

// ---------------------------------------------------------------------------
// Stable grouping of a decode call with at most 64 routed pairs (one per
// lane), in registers.  For the pair p of lane p with expert e: eq = the
// pairs of the same expert and lo = the pairs of a lower expert, from one
// ballot per bit of the expert index (most significant first).  Then the
// pair's position is |lo| + (earlier pairs in eq), and its group's index
// among the non-empty routed groups is the number of group leaders (first
// pairs) in lo.  The order is the one permute_decode_wave produces.
// ---------------------------------------------------------------------------
constexpr int kDecodeSmallPairs = 64;

__device__ __forceinline__ void pair_masks(bool ok, int e, int E, uint64_t& eq, uint64_t& lo) {
  const int nbits = E > 1 ? 32 - __builtin_clz((unsigned)(E - 1)) : 0;
  eq = __ballot(ok);
  lo = 0;
  for (int b = nbits - 1; b >= 0; --b) {
    const bool bit = (e >> b) & 1;
    const uint64_t ones = __ballot(ok && bit);
    if (bit) lo |= eq & ~ones;
    eq &= bit ? ones : ~ones;
  }
  if (!ok) eq = lo = 0;
}

__device__ __forceinline__ int wave_or(int v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v |= __shfl_xor(v, o, 64);
  return v;
}

// DecodeWork descriptors and the residency status of a call with T*k <= 64
// pairs (one wave): what the expert kernels read.  Positions i >= n of a
// descriptor are left as they were (the kernels read only i < n).
__device__ inline void decode_work_small(const int32_t* idx_s, const float* w_s, const int* xe_s,
                                         const int* slot_s, int T, int k, int E, int S,
                                         const ExpertPool& ep, DecodeWork* __restrict__ work,
                                         int max_active) {
  const int lane = threadIdx.x & 63;
  const int P = T * k;
  const bool ok = lane < P;
  const int e = ok ? idx_s[lane] : 0;
  const float w = ok ? w_s[lane] : 0.f;
  uint64_t eq, lo;
  pair_masks(ok, e, E, eq, lo);
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int rank = __popcll(eq & lt);
  const bool lead = ok && rank == 0;
  const uint64_t leaders = __ballot(lead);
  const int a = __popcll(lo & leaders), nr = __popcll(leaders);
  int bits = 0;
  if (lead) {
    const int slot = slot_s[e];
    bits |= slot < 0 ? 1 : (slot >= ep.n_slots ? 2 : 0);
    DecodeWork* wk = work + a;
    wk->group = e;
    wk->slot = slot;
    wk->off = __popcll(lo);
    wk->n = __popcll(eq);
  }
  if (ok) {
    const int t = lane / k;
    DecodeWork* wk = work + a;
    wk->tok[rank] = t;
    wk->xe[rank] = xe_s[t];
    wk->w[rank] = w;
  }
  // shared experts follow the routed groups: every token in order, weight 1
  for (int s = lane; s < S; s += 64) {
    const int slot = slot_s[E + s];
    bits |= slot < 0 ? 1 : (slot >= ep.n_slots ? 2 : 0);
    DecodeWork* wk = work + nr + s;
    wk->group = E + s;
    wk->slot = slot;
    wk->off = P + s * T;
    wk->n = T;
  }
  for (int i = lane; i < S * T; i += 64) {
    const int s = i / T, t = i - s * T;
    DecodeWork* wk = work + nr + s;
    wk->tok[t] = t;
    wk->xe[t] = xe_s[t];
    wk->w[t] = 1.0f;
  }
  for (int aa = nr + S + lane; aa < max_active; aa += 64) work[aa].group = -1;
  bits = wave_or(bits);
  if (lane == 0 && ep.status) *ep.status = bits;
}

// DecodeWork descriptors and the residency status of a one-token call with
// E <= 64 experts and k + S <= 64 groups (one wave), straight from the
// selection in registers: the selected experts in expert order (group a at
// position a, one pair each), then the shared experts.  xe: the token's
// fixed-point exponent.  The same descriptors as decode_work_small.
__device__ inline void decode_work_one_token(const float* lgrow, int E, int k, int S,
                                             int softmax_all, int xe, const int* slot_s,
                                             const ExpertPool& ep, DecodeWork* __restrict__ work,
                                             int max_active) {
  const int lane = threadIdx.x & 63;
  bool sel;
  int rank;
  float w;
  topk_lane64(lgrow, E, k, softmax_all, sel, rank, w);
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int a = __popcll(__ballot(sel) & lt);
  int bits = 0;
  if (sel) {
    const int slot = slot_s[lane];
    bits = slot < 0 ? 1 : (slot >= ep.n_slots ? 2 : 0);
    DecodeWork* wk = work + a;
    wk->group = lane;
    wk->slot = slot;
    wk->off = a;
    wk->n = 1;
    wk->tok[0] = 0;
    wk->xe[0] = xe;
    wk->w[0] = w;
  }
  if (lane < S) {
    const int slot = slot_s[E + lane];
    bits = slot < 0 ? 1 : (slot >= ep.n_slots ? 2 : 0);
    DecodeWork* wk = work + k + lane;
    wk->group = E + lane;
    wk->slot = slot;
    wk->off = k + lane;
    wk->n = 1;
    wk->tok[0] = 0;
    wk->xe[0] = xe;
    wk->w[0] = 1.0f;
  }
  for (int aa = k + S + lane; aa < max_active; aa += 64) work[aa].group = -1;
  const int st = (__ballot(bits & 1) ? 1 : 0) | (__ballot(bits & 2) ? 2 : 0);
  if (lane == 0 && ep.status) *ep.status = st;
}

// The caller's optional routing outputs of a call with T*k <= 64 pairs (one
// wave, beside decode_work_small): top-k, permutation order, group counts
// and offsets.  cnt_s: LDS scratch of E ints.
__device__ inline void decode_outputs_small(const int32_t* idx_s, const float* w_s, int T, int k,
                                            int E, int S, const PermOut& o, int* cnt_s) {
  const int lane = threadIdx.x & 63;
  const int P = T * k, G = E + S;
  const bool ok = lane < P;
  const int e = ok ? idx_s[lane] : 0;
  if (ok) {
    if (o.idx_out) o.idx_out[lane] = e;
    if (o.w_out) o.w_out[lane] = w_s[lane];
  }
  if (!o.order_out && !o.counts_out && !o.offsets_out) return;
  uint64_t eq, lo;
  pair_masks(ok, e, E, eq, lo);
  const uint64_t lt = lane ? (~0ull >> (64 - lane)) : 0ull;
  const int rank = __popcll(eq & lt);
  if (o.order_out) {
    if (ok) o.order_out[__popcll(lo) + rank] = lane;
    for (int i = lane; i < S * T; i += 64) o.order_out[P + i] = P + i;
  }
  if (!o.counts_out && !o.offsets_out) return;
  for (int g = lane; g < E; g += 64) cnt_s[g] = 0;
  __builtin_amdgcn_wave_barrier();
  if (ok && rank == 0) cnt_s[e] = __popcll(eq);
  __builtin_amdgcn_wave_barrier();
  // exclusive scan over groups, 4 consecutive groups per lane
  int c4[4], sum = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int g = lane * 4 + i;
    c4[i] = g < E ? cnt_s[g] : (g < G ? T : 0);
    sum += c4[i];
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
      if (o.counts_out) o.counts_out[g] = c4[i];
      if (o.offsets_out) o.offsets_out[g] = run;
    }
    run += c4[i];
  }
  if (lane == 63 && o.offsets_out) o.offsets_out[G] = incl;
}

inline PermOut perm_out(const WsPtr& w, int32_t* counts_out, int32_t* idx_out, float* wts_out,
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

}  // namespace mira
