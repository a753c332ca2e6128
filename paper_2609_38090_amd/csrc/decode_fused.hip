// Decode gate/up with the routing done in the same kernel.
//
// For calls of at most five tokens every workgroup of the gate/up grid runs
// the router itself (logits with the arithmetic of the routing kernels, so
// the choice of experts is bit-identical to the other paths; top-k and
// combine weights, section II-A), finds the expert group it serves, writes
// the fixed-point digits of that group's tokens into LDS and then streams its
// 64 rows of the packed gate and up matrices through the int8 matrix cores
// (body in decode_dev.h).  Workgroup 0 also writes the full routing (the
// descriptors the down kernel reads and every optional output).  The
// separate preparation launch and its dependency on the expert kernels
// disappear from the one-shot forward call.
#include "decode_dev.h"
#include "route_dev.h"

namespace mira {

constexpr int kFusedThreads = 256;
constexpr int kFusedWaves = kFusedThreads / 64;
constexpr int kFusedMaxTok = kTokPerGroup;          // one 16-column digit operand
constexpr int kFusedMaxDynLds = 64 * 1024;          // digits (or logit partials) in LDS
constexpr int kPartBytes = kBigWaves * 16 * 17 * 4;  // logit partials of 16 k-range slices
constexpr int kTouchLoads = 8;  // 128-byte lines per thread touched ahead of the router (256 KB)

// Bytes of the dynamic LDS region: the logit partials during routing, then
// the digits of up to T tokens, [T][3][C + 16] int8 (rows padded by 16 bytes
// so the 15 digit rows of one read phase fall on distinct banks).
static size_t fused_dyn_lds(int T, int C) {
  const size_t dig = (size_t)T * kDigits * (C + 16);
  return dig > (size_t)kPartBytes ? dig : (size_t)kPartBytes;
}

bool decode_fused_ok(const Layout& L) {
  return L.T >= 1 && L.T <= kFusedMaxTok && fused_dyn_lds(L.T, L.C) <= (size_t)kFusedMaxDynLds;
}

template <typename ActT>
__global__ __launch_bounds__(kFusedThreads) void decode_route_gateup_kernel(
    int C, int R, int T, int E, int k, int S, int softmax_all, const ActT* __restrict__ x,
    const ActT* __restrict__ wr, const float* __restrict__ bias, float* __restrict__ logits_out,
    ExpertPool ep, PermOut o, DecodeWork* __restrict__ work, int max_active,
    int8_t* __restrict__ hdig, int32_t* __restrict__ hexp) {
  extern __shared__ __attribute__((aligned(16))) int8_t dyn_s[];
  __shared__ float lg[kFusedMaxTok][MIRA_MAX_EXPERTS];
  __shared__ float bias_s[MIRA_MAX_EXPERTS];
  __shared__ int slot_s[MIRA_MAX_EXPERTS];
  __shared__ int32_t idx_s[kFusedMaxTok * MIRA_MAX_TOPK];
  __shared__ float w_s[kFusedMaxTok * MIRA_MAX_TOPK];
  __shared__ int sel_e[kFusedWaves][MIRA_MAX_TOPK];
  __shared__ float sel_v[kFusedWaves][MIRA_MAX_TOPK];
  __shared__ float xmax_s[kRouteTok];
  __shared__ int xe_s[kFusedMaxTok];
  __shared__ int cnt_s[MIRA_MAX_EXPERTS], run_s[MIRA_MAX_EXPERTS];
  __shared__ int ptok_s[kDecodeMaxPairs];
  __shared__ float pw_s[kDecodeMaxPairs];
  __shared__ int grp_s[4];  // group, offset, tokens, number of non-empty groups
  __shared__ int gtok_s[kFusedMaxTok];
  __shared__ float bmax[4][kTokPerGroup];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int G = E + S;

  // Touch every 128-byte line of the router rows and of x once, up front:
  // the k-range slices below then wait for memory once instead of once per
  // slice.  The loaded words are folded into a value that is consumed after
  // the logits (and never stored, as T >= 1).
  uint32_t touch = 0;
  {
    const size_t wbytes = (size_t)E * C * sizeof(ActT), xbytes = (size_t)T * C * sizeof(ActT);
    uint32_t tv[kTouchLoads];
#pragma unroll
    for (int i = 0; i < kTouchLoads; ++i) {
      const size_t off = ((size_t)i * kFusedThreads + tid) * 128;
      tv[i] = off < wbytes ? *(const uint32_t*)((const char*)wr + off)
              : off - wbytes < xbytes ? *(const uint32_t*)((const char*)x + (off - wbytes)) : 0u;
    }
#pragma unroll
    for (int i = 0; i < kTouchLoads; ++i) touch |= tv[i];
  }

  for (int e = tid; e < G; e += kFusedThreads) {
    if (e < E) bias_s[e] = bias ? bias[e] : 0.f;
    slot_s[e] = ep.slot_table[e];  // read now: the table may change after the call is queued
  }
  __syncthreads();

  // router logits and max |x| per token
  float(*lgp)[MIRA_MAX_EXPERTS] = lg;
  if constexpr (sizeof(ActT) == 2) {
    logits_slices_bf16<kFusedWaves>(x, wr, bias ? bias_s : nullptr, T, E, C,
                                    (float(*)[16][17])dyn_s, lgp, xmax_s);
  } else {
    logits_tile_f32(x, wr, bias, T, E, C, 0, kFusedWaves, lgp);
    for (int t = wave; t < T; t += kFusedWaves) {
      float m = 0.f;
      for (int c = lane * 4; c < C; c += 256) {
        float v[4];
        load4_act(x + (size_t)t * C + c, v);
        m = fmaxf(m, fmaxf(fmaxf(fabsf(v[0]), fabsf(v[1])), fmaxf(fabsf(v[2]), fabsf(v[3]))));
      }
      m = wave_max(m);
      if (lane == 0) xmax_s[t] = m;
    }
    __syncthreads();
  }
  // top-k and combine weights, one wave per token
  for (int t = wave; t < T; t += kFusedWaves) {
    if (logits_out && blockIdx.x == 0)
      for (int e = lane; e < E; e += 64) logits_out[(size_t)t * E + e] = lg[t][e];
    topk_rank(lg[t], E, k, softmax_all, idx_s + t * k, w_s + t * k, sel_e[wave], sel_v[wave]);
  }
  if (tid < T) xe_s[tid] = kFixBits - exp_bound(xmax_s[tid]);
  if (T < 0) hexp[tid] = (int32_t)touch;  // keeps the touch loads; never taken
  __syncthreads();

  // workgroup 0, wave 0: the routing every later kernel and the caller read
  if (blockIdx.x == 0 && wave == 0)
    permute_decode_wave(idx_s, w_s, xe_s, slot_s, T, k, E, S, ep, o, work, max_active, cnt_s,
                        run_s, ptok_s, pw_s);

  // wave 1: the expert group a = blockIdx.x / nrb of this workgroup (the a-th
  // non-empty group, routed experts then shared), its first position in the
  // permuted order and its tokens in pair order
  const int nrb = R / kBlk;
  const int a = blockIdx.x / nrb, rb = blockIdx.x - a * nrb;
  if (wave == 1) {
    const int Tk = T * k;
    int c4[4], sum = 0, nz = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = lane * 4 + i;
      c4[i] = (g >= E && g < G) ? T : 0;
    }
    for (int p = 0; p < Tk; ++p) {
      const int e = idx_s[p];
#pragma unroll
      for (int i = 0; i < 4; ++i) c4[i] += (e == lane * 4 + i);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sum += c4[i];
      nz += c4[i] > 0;
    }
    int incl = sum, inz = nz;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off, 64), vz = __shfl_up(inz, off, 64);
      if (lane >= off) {
        incl += v;
        inz += vz;
      }
    }
    int run = incl - sum, rank = inz - nz;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (c4[i] > 0) {
        if (rank == a) {
          grp_s[0] = lane * 4 + i;
          grp_s[1] = run;
          grp_s[2] = c4[i];
        }
        ++rank;
      }
      run += c4[i];
    }
    if (lane == 63) grp_s[3] = inz;
  }
  __syncthreads();
  if (a >= grp_s[3]) return;  // fewer non-empty groups than the grid provides for
  const int g = grp_s[0], off = grp_s[1], n = grp_s[2];
  if (wave == 1) {
    if (g >= E) {
      if (lane < n) gtok_s[lane] = lane;
    } else {
      const int Tk = T * k;
      const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
      int base = 0;
      for (int p0 = 0; p0 < Tk; p0 += 64) {
        const int p = p0 + lane;
        const bool hit = p < Tk && idx_s[p] == g;
        const uint64_t mask = __ballot(hit);
        if (hit) gtok_s[base + __popcll(mask & lt_mask)] = p / k;
        base += __popcll(mask);
      }
    }
  }
  __syncthreads();

  // fixed-point digits of the group's tokens (|x * 2^E_t| < 2^22 per token)
  const int CP = C + 16;
  for (int i = tid; i < n * (C / 4); i += kFusedThreads) {
    const int j = i / (C / 4), c = (i - j * (C / 4)) * 4;
    const int t = gtok_s[j], Ex = xe_s[t];
    float v[4];
    load4_act(x + (size_t)t * C + c, v);
    uint32_t w0 = 0, w1 = 0, w2 = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      int d0, d1, d2;
      split_digits((int)rintf(ldexpf(v[q], Ex)), d0, d1, d2);
      w0 |= (uint32_t)(d0 & 0xFF) << (8 * q);
      w1 |= (uint32_t)(d1 & 0xFF) << (8 * q);
      w2 |= (uint32_t)(d2 & 0xFF) << (8 * q);
    }
    int8_t* dst = dyn_s + (size_t)j * kDigits * CP + c;
    *(uint32_t*)(dst) = w0;
    *(uint32_t*)(dst + CP) = w1;
    *(uint32_t*)(dst + 2 * CP) = w2;
  }
  __syncthreads();

  const int slot = slot_s[g];
  if (slot < 0 || slot >= ep.n_slots) {
    if (tid == 0 && ep.status) atomicOr(ep.status, slot < 0 ? 1 : 2);
    return;
  }
  const int r16 = lane & 15, kg = lane >> 4;
  const int m = r16 / 3, d = r16 - 3 * m;
  bool bv[1];
  int xev[1];
  bv[0] = r16 < 3 * kTokPerGroup && m < n;
  xev[0] = bv[0] ? xe_s[gtok_s[m]] : 0;
  const int8_t* xdl = dyn_s + (size_t)((bv[0] ? m : 0) * kDigits + d) * CP + kg * 16;
  gateup_block<1>(C, R, rb, ep.pool + (size_t)slot * ep.stride, off, bv, xev,
                  [&](int, int ks) { return *(const v4i*)(xdl + ks * 64); }, hdig, hexp, bmax);
}

hipError_t launch_decode_fused(const mira_shape& s, const Layout& L, const WsPtr& w,
                               const void* x, const void* wr, const float* bias, float* logits_out,
                               const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                               float* wts_out, int32_t* offsets_out, int32_t* order_out,
                               float* out, hipStream_t st) {
  if (L.T == 0) return hipSuccess;
  const int sa = (s.flags & MIRA_FLAG_SOFTMAX_ALL) ? 1 : 0;
  const PermOut o = perm_out(w, counts_out, idx_out, wts_out, offsets_out, order_out);
  const int max_active = decode_max_active(L);
  const dim3 grid(max_active * (L.R / kBlk)), block(kFusedThreads);
  const uint32_t dyn = (uint32_t)fused_dyn_lds(L.T, L.C);
  if (s.act_dtype == MIRA_BF16)
    launch_timed("decode_route_gateup", decode_route_gateup_kernel<uint16_t>, grid, block, dyn, st,
                 L.C, L.R, L.T, L.E, L.k, L.S, sa, (const uint16_t*)x, (const uint16_t*)wr, bias,
                 logits_out, ep, o, w.dwork, max_active, w.hdig, w.hexp);
  else
    launch_timed("decode_route_gateup", decode_route_gateup_kernel<float>, grid, block, dyn, st,
                 L.C, L.R, L.T, L.E, L.k, L.S, sa, (const float*)x, (const float*)wr, bias,
                 logits_out, ep, o, w.dwork, max_active, w.hdig, w.hexp);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_decode_down(L, w, ep, out, st);
}

}  // namespace mira
