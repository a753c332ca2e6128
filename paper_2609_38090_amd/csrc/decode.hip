// Small-batch (decode) expert FFN over packed experts: gate/up + SwiGLU
// (body in decode_dev.h) and the down projection with the weighted combine.
//
// With one to a few tokens per expert the step is bound by streaming the
// packed int8 bytes from HBM.  Both kernels feed those bytes unchanged to the
// int8 matrix cores (v_mfma_i32_16x16x64_i8): the activation side is written
// as a fixed-point integer split into signed base-256 digits, each digit one
// int8 operand column, so the products and sums are exact int32 and the only
// rounding is the fixed-point step and the final fp32 arithmetic.  x has three
// digits (2^-22 of the token's maximum); H' three (2^-22 of its 64-row block
// maximum) when the call has at most 5 tokens, else two (2^-14).  A one-token
// call instead gives every 16-row tile of H' its own exponent (three digits):
// its gate/up splits the tiles evenly over the CUs, and its down kernel gives
// each (tile, digit) pair of a k-step its own operand column.  Since the
// shared scale sigma_r factors out (section IV-B), y = Qd H' with
// H' = sigma (.) silu(G) (.) U.
#include "decode_dev.h"

namespace mira {

// ---------------------------------------------------------------------------
// Gate/up + SwiGLU of calls with several tokens.  Workgroup = (non-empty
// expert a, block of 64 rows of R); the digits of x come from the workspace
// (xdig[(t*3 + d)*C + c], written by the decode preparation kernel).
// ---------------------------------------------------------------------------
// With XL (INT4, one token group, C <= kXlMaxC) the workgroup first copies
// the digit rows of its tokens into LDS (row stride C + 16 bytes, so the 16
// rows a read phase touches fall in distinct banks) and the loop reads them
// from there.
constexpr int kXlMaxC = 4096;
constexpr int kXlUnroll = 16;  // k-steps per weight batch
// k-steps per weight batch of the one-token INT4 tile kernel (6 KB per wave):
// a wave holds one tile and cannot issue its next loads while it unpacks and
// scales a batch, and shorter batches measured faster than 4, 8 or 16 steps
constexpr int kTileI4Unroll = 6;

template <int NG, bool I4, bool XL>
__device__ __forceinline__ void decode_gateup_body(int C, int R, const ExpertPool& ep,
                                                   DecodeWork* __restrict__ work,
                                                   const int8_t* __restrict__ xdig,
                                                   int8_t* __restrict__ hdig,
                                                   int32_t* __restrict__ hexp) {
  __shared__ float bmax[4][NG * kTokPerGroup];
  const int nrb = R / kBlk;
  const int a = blockIdx.x / nrb, rb = blockIdx.x - a * nrb;
  const DecodeWork& wk = work[a];
  const int g = wk.group;
  if (g < 0) return;
  const int slot = ep.slot_table[g];  // read now: the table may change after routing
  const bool ok = slot >= 0 && slot < ep.n_slots;
  // block 0 of the expert keeps the resolved slot for the down kernel
  if (rb == 0 && threadIdx.x == 0) work[a].slot = ok ? slot : -1;
  if (!ok) {
    if (threadIdx.x == 0 && ep.status) atomicOr(ep.status, slot < 0 ? 1 : 2);
    return;
  }
  const int n = wk.n;
  const int lane = threadIdx.x & 63;
  const int r16 = lane & 15, kg = lane >> 4;
  const int m = r16 / 3, d = r16 - 3 * m;
  const int8_t* bp[NG];
  bool bv[NG];
  int xev[NG];
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    const int i = cg * kTokPerGroup + m;
    bv[cg] = r16 < 3 * kTokPerGroup && i < n;
    const int tok = bv[cg] ? wk.tok[i] : 0;
    xev[cg] = bv[cg] ? wk.xe[i] : 0;
    bp[cg] = xdig + ((size_t)tok * kDigits + d) * C + kg * 16;
  }
  if constexpr (XL) {
    static_assert(NG == 1, "one token group in LDS");
    __shared__ __attribute__((aligned(16))) int8_t xl[16 * (kXlMaxC + 16)];
    const int ld = C + 16;
    const int chunks = C / 16;
    // only the digit rows of the group's tokens are staged; lanes of the
    // other columns take a zero operand without reading LDS
    const int rows = 3 * min(n, kTokPerGroup);
    for (int i = threadIdx.x; i < rows * chunks; i += 256) {
      const int row = i / chunks, c16 = i - row * chunks;
      const int cg = row >> 4, col = row & 15;
      const int mm = col / 3, dd = col - 3 * mm, ti = cg * kTokPerGroup + mm;
      v4i v = zero16();
      if (col < 3 * kTokPerGroup && ti < n)
        v = ld16(xdig + ((size_t)wk.tok[ti] * kDigits + dd) * C + c16 * 16);
      *(v4i*)(xl + (size_t)row * ld + c16 * 16) = v;
    }
    __syncthreads();
    const int8_t* xr[NG];
#pragma unroll
    for (int cg = 0; cg < NG; ++cg) xr[cg] = xl + (size_t)(cg * 16 + r16) * ld + kg * 16;
    const auto load_x = [&](int cg, int ks) { return bv[cg] ? *(const v4i*)(xr[cg] + ks * 64) : zero16(); };
    gateup_block_i4<NG, kXlUnroll, true>(C, R, rb, (const uint8_t*)ep.pool + (size_t)slot * ep.stride,
                                         wk.off, bv, xev, load_x, hdig, hexp, bmax);
    return;
  }
  const auto load_b = [&](int cg, int ks) { return ld16(bp[cg] + ks * 64); };
  if constexpr (I4)
    gateup_block_i4<NG, dec_unroll(NG), false>(C, R, rb,
                                               (const uint8_t*)ep.pool + (size_t)slot * ep.stride,
                                               wk.off, bv, xev, load_b, hdig, hexp, bmax);
  else
    gateup_block<NG>(C, R, rb, ep.pool + (size_t)slot * ep.stride, wk.off, bv, xev, load_b, hdig,
                     hexp, bmax);
}

template <int NG, bool I4>
__global__ __launch_bounds__(256) void decode_gateup_kernel(int C, int R, ExpertPool ep,
                                                            DecodeWork* __restrict__ work,
                                                            const int8_t* __restrict__ xdig,
                                                            int8_t* __restrict__ hdig,
                                                            int32_t* __restrict__ hexp) {
  decode_gateup_body<NG, I4, false>(C, R, ep, work, xdig, hdig, hexp);
}

// The LDS variant keeps two workgroups per CU (the 64 KB of digits each).
__global__ __launch_bounds__(256, 2) void decode_gateup_xl_kernel(int C, int R, ExpertPool ep,
                                                                 DecodeWork* __restrict__ work,
                                                                 const int8_t* __restrict__ xdig,
                                                                 int8_t* __restrict__ hdig,
                                                                 int32_t* __restrict__ hexp) {
  decode_gateup_body<1, true, true>(C, R, ep, work, xdig, hdig, hexp);
}

// One-token calls: every wave streams one 16-row tile of the concatenated
// rows of the active experts (tile t = expert a, rows 16*(t mod R/16) ..)
// and writes that tile's H' with its own exponent (h_tile_1tok), so no wave
// waits for another and the host splits the tiles evenly over the CUs (W
// waves per workgroup, about one workgroup per CU).  The wave of tile 0 of
// each expert also stores the slot it resolved from the table in the
// expert's descriptor (-1 if invalid), for the down kernel.
constexpr int kTileMaxWaves = 8;

__global__ __launch_bounds__(64 * kTileMaxWaves) void decode_gateup_tile_kernel(
    int C, int R, int W, int ntiles, ExpertPool ep, DecodeWork* __restrict__ work,
    const int8_t* __restrict__ xdig, int8_t* __restrict__ hdig, int32_t* __restrict__ hexp) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t = blockIdx.x * W + wave;
  if (wave >= W || t >= ntiles) return;
  const int tpe = R / 16;
  const int a = t / tpe, rt = t - a * tpe;
  const DecodeWork& wk = work[a];
  const int g = wk.group;
  if (g < 0) return;
  const int slot = ep.slot_table[g];  // read now: the table may change after routing
  const bool ok = slot >= 0 && slot < ep.n_slots;
  if (rt == 0 && lane == 0) work[a].slot = ok ? slot : -1;
  if (!ok) {
    if (lane == 0 && ep.status) atomicOr(ep.status, slot < 0 ? 1 : 2);
    return;
  }
  const int r16 = lane & 15, kg = lane >> 4;
  const bool bv = r16 < 3 && wk.n > 0;
  const int tok = bv ? wk.tok[0] : 0;
  const int xe = bv ? wk.xe[0] : 0;
  const int8_t* bp = xdig + ((size_t)tok * kDigits + (bv ? r16 : 0)) * C + kg * 16;
  const auto load_b = [&](int, int ks) { return ld16(bp + ks * 64); };
  // seven 16-row tiles per CU at Mixtral's shape: one wave per tile beat two
  // waves per tile (gate and up streamed apart, up sums handed over in LDS)
  // by 0.45 us per call
  v4i accg[1], accu[1];
  float sg[4];
  const bool bva[1] = {bv};
  gateup_tile_stream<1>(C, R, rt, ep.pool + (size_t)slot * ep.stride, bva, load_b, accg, accu, sg);
  h_tile_1tok(R, rt, wk.off, bv, xe, accg[0], accu[0], sg, hdig, hexp);
}

// One-token INT4 calls (C <= kXlMaxC): the same tile split, with the
// token's three digit rows copied into LDS once per workgroup (row stride
// C + 16 bytes), so a wave's batches hold only weight registers.  A one-token
// call's only token is token 0, whatever expert a tile belongs to.
__global__ __launch_bounds__(64 * kTileMaxWaves) void decode_gateup_tile_i4_kernel(
    int C, int R, int W, int ntiles, ExpertPool ep, DecodeWork* __restrict__ work,
    const int8_t* __restrict__ xdig, int8_t* __restrict__ hdig, int32_t* __restrict__ hexp) {
  __shared__ __attribute__((aligned(16))) int8_t xl[kDigits * (kXlMaxC + 16)];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int ld = C + 16, chunks = C / 16;
  for (int i = threadIdx.x; i < kDigits * chunks; i += blockDim.x) {
    const int row = i / chunks, c16 = i - row * chunks;
    *(v4i*)(xl + (size_t)row * ld + c16 * 16) = ld16(xdig + (size_t)row * C + c16 * 16);
  }
  __syncthreads();
  const int t = blockIdx.x * W + wave;
  if (wave >= W || t >= ntiles) return;
  const int tpe = R / 16;
  const int a = t / tpe, rt = t - a * tpe;
  const DecodeWork& wk = work[a];
  const int g = wk.group;
  if (g < 0) return;
  const int slot = ep.slot_table[g];  // read now: the table may change after routing
  const bool ok = slot >= 0 && slot < ep.n_slots;
  if (rt == 0 && lane == 0) work[a].slot = ok ? slot : -1;
  if (!ok) {
    if (lane == 0 && ep.status) atomicOr(ep.status, slot < 0 ? 1 : 2);
    return;
  }
  const int r16 = lane & 15, kg = lane >> 4;
  const bool bv = r16 < 3 && wk.n > 0;
  const int xe = bv ? wk.xe[0] : 0;
  const int8_t* xr = xl + (size_t)(bv ? r16 : 0) * ld + kg * 16;
  const auto load_x = [&](int, int ks) { return bv ? *(const v4i*)(xr + ks * 64) : zero16(); };
  float accg[1][4], accu[1][4];
  const bool bva[1] = {bv};
  gateup_tile_stream_i4<1, kTileI4Unroll, true>(C, R, rt, (const uint8_t*)ep.pool + (size_t)slot * ep.stride,
                                                bva, load_x, accg, accu);
  // 2^-E of the token's fixed point, and 1/16 for the nibble operand (16*q)
  const bool lead = bv && r16 == 0;
  const float xs = bv ? ldexpf(1.f, -xe - 4) : 0.f;
  float hv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float gv = combine_digits_f(accg[0][i]) * xs;
    const float uv = combine_digits_f(accu[0][i]) * xs;
    const float h = gv / (1.f + expf(-gv)) * uv;
    hv[i] = lead ? h : 0.f;
  }
  write_h_tile_1tok(R, rt, wk.off, lead, hv, hdig, hexp);
}

// ---------------------------------------------------------------------------
// Down projection + weighted combine.  Workgroup = 16 output rows c; its KS
// waves split the R dimension.  For every non-empty expert, y = Qd H' with
// per-64-row exponents of H', multiplied by the combine weight of each
// (token, expert) pair and summed per token in a fixed order (expert list
// order inside a wave, then wave order), so the result is deterministic.
// H' has HD digits per entry (h_digits): an operand of 16 columns holds 5
// tokens of three digits or 8 of two (column r16 = token r16/HD of the
// group, digit r16%HD), and NG groups cover that many tokens per group.
// ---------------------------------------------------------------------------
template <int NG, int KS, bool I4, int HD, bool TE>
__global__ __launch_bounds__(64 * KS) void decode_down_kernel(
    int C, int R, int T, int max_active, ExpertPool ep, const DecodeWork* __restrict__ work,
    const int8_t* __restrict__ hdig, const int32_t* __restrict__ hexp, float* __restrict__ out) {
  constexpr int TPG = h_tok_per_group(HD);
  __shared__ float part[KS][MIRA_DECODE_MAX_TOKENS][16];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // each wave adds only into its own slice, so it clears only that slice and
  // nothing waits before the stream starts
  for (int i = lane; i < MIRA_DECODE_MAX_TOKENS * 16; i += 64) (&part[wave][0][0])[i] = 0.f;

  static_assert(!TE || (NG == 1 && HD == 3), "per-tile exponents: one token, three digits");
  const int r16 = lane & 15, kg = lane >> 4;
  // TE: column r16 < 12 is digit d of the k-step's tile j = r16/3 (k group
  // j), so each tile's digits carry their own exponent; otherwise column
  // r16 is digit d of token m
  const int m = r16 / HD, d = r16 - HD * m;
  const int nks = R / 64;
  // k-steps per wave; even for INT4, whose loads cover two k-steps
  const int spw = I4 ? (((nks + KS - 1) / KS + 1) & ~1) : (nks + KS - 1) / KS;
  const int ks_beg = wave * spw, ks_end = min(nks, ks_beg + spw);

  for (int a = 0; a < max_active; ++a) {
    const DecodeWork& wk = work[a];
    if (wk.group < 0) break;
    // the slot the gate/up kernel resolved from the table (-1 if invalid)
    const int slot = wk.slot;
    if (slot < 0 || slot >= ep.n_slots) continue;
    const int off = wk.off, n = wk.n;
    // tile row c0/16 of the down matrix: INT8 tiles of 1 KB (lane l at 16*l),
    // or INT4 nibble tiles of two groups (lane l at 16*l) and the tile-row's
    // 32-byte scale blocks (lane l at 8*l of a 16-group run)
    const int8_t* base = ep.pool + (size_t)slot * ep.stride;
    const int8_t* dp = I4 ? base + 2 * i4_matrix_bytes(R, C) + (size_t)blockIdx.x * (nks / 2) * kI4PairTile +
                                lane * 16
                          : base + (size_t)2 * R * C + (size_t)blockIdx.x * nks * 1024 + lane * 16;
    const int8_t* sp = base + 2 * i4_matrix_bytes(R, C) + i4_nib_bytes(C, R) +
                       (size_t)blockIdx.x * nks * 32 + lane * 8;
    const int8_t* bp[NG];
    const int32_t* hx[NG];
    bool bv[NG];
#pragma unroll
    for (int cg = 0; cg < NG; ++cg) {
      const int i = TE ? 0 : cg * TPG + m;
      bv[cg] = (TE ? r16 < 12 : r16 < HD * TPG) && i < n;
      const size_t pos = (size_t)off + (bv[cg] ? i : 0);
      bp[cg] = hdig + (pos * HD + d) * R + kg * 16;
      hx[cg] = TE ? hexp + pos * (R / 16) + m : hexp + pos * nks;
    }
    // TE: only the lanes of k group j load their tile's digits
    const bool bload = !TE || kg == m;
    // the combine's token and weight, loaded ahead of the stream so that
    // they return with the first batch
    int ctok[NG];
    float cwgt[NG];
#pragma unroll
    for (int cg = 0; cg < NG; ++cg) {
      const bool lead = (TE ? r16 == 0 : d == 0) && bv[cg];
      const int ti = TE ? 0 : cg * TPG + m;
      ctok[cg] = lead ? wk.tok[ti] : 0;
      cwgt[cg] = lead ? wk.w[ti] : 0.f;
    }
    float facc[NG][4];
#pragma unroll
    for (int cg = 0; cg < NG; ++cg)
#pragma unroll
      for (int i = 0; i < 4; ++i) facc[cg][i] = 0.f;

    // k-steps per batch: with 14 or 16 waves (up to four per SIMD, at most
    // 128 registers each) half the batch of the 8-wave layout
    static_assert(KS > 8, "the batch size assumes more than 8 waves");
    constexpr int kDecUnroll = dec_unroll(NG) / 2;
    static_assert(kDecUnroll % 2 == 0 && kDecUnroll <= 16, "INT4 batches cover whole tiles");
    struct Batch {
      v4i a[I4 ? kDecUnroll / 2 : kDecUnroll], b[kDecUnroll][NG];
      uint2 s4;  // INT4: lane l holds group ks0 + l/4, rows 4*(l%4) .. +3
      int he[kDecUnroll][NG];
    };
    auto issue = [&](Batch& bt, int ks0) {
      if constexpr (I4) {
#pragma unroll
        for (int p = 0; p < kDecUnroll / 2; ++p) {
          const bool in = ks0 + 2 * p < ks_end;
          bt.a[p] = in ? ld16_stream(dp + (size_t)(ks0 / 2 + p) * kI4PairTile) : zero16();
        }
        const bool sin = (lane >> 2) < kDecUnroll && ks0 + (lane >> 2) < ks_end;
        bt.s4 = sin ? ld8_stream(sp + (size_t)ks0 * 32) : uint2{0, 0};
      }
#pragma unroll
      for (int u = 0; u < kDecUnroll; ++u) {
        const int ks = ks0 + u;
        const bool in = ks < ks_end;
        if constexpr (!I4) bt.a[u] = in ? ld16_stream(dp + ks * 1024) : zero16();
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) {
          bt.b[u][cg] = (in && bv[cg] && bload) ? ld16(bp[cg] + ks * 64) : zero16();
          bt.he[u][cg] = (in && bv[cg]) ? hx[cg][TE ? 4 * ks : ks] : 0;
        }
      }
    };
    auto consume = [&](const Batch& bt) {
#pragma unroll
      for (int u = 0; u < kDecUnroll; ++u) {
        v4i a;
        float s4[4] = {1.f, 1.f, 1.f, 1.f};
        if constexpr (I4) {
          const v4i q2 = bt.a[u / 2];
          a = (u & 1) ? i4_operand(uint2{(uint32_t)q2[2], (uint32_t)q2[3]})
                      : i4_operand(uint2{(uint32_t)q2[0], (uint32_t)q2[1]});
          i4_scales(uint2{(uint32_t)__shfl((int)bt.s4.x, 4 * u + kg, 64),
                          (uint32_t)__shfl((int)bt.s4.y, 4 * u + kg, 64)}, s4);
        } else {
          a = bt.a[u];
        }
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) {
          const v4i sres = mfma_i8(a, bt.b[u][cg], zero16());
          // digit weight and H' exponent; INT4 adds the row scales and 1/16
          const float sc = bv[cg] ? ldexpf(1.f, 8 * d - bt.he[u][cg] - (I4 ? 4 : 0)) : 0.f;
#pragma unroll
          for (int i = 0; i < 4; ++i) facc[cg][i] = fmaf((float)sres[i], sc * s4[i], facc[cg][i]);
        }
      }
    };
    // one batch per iteration (see the gate/up body)
    for (int ks = ks_beg; ks < ks_end; ks += kDecUnroll) {
      Batch bt;
      issue(bt, ks);
      consume(bt);
    }
#pragma unroll
    for (int cg = 0; cg < NG; ++cg) {
      const bool lead = (TE ? r16 == 0 : d == 0) && bv[cg];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float v;
        if constexpr (TE) {
          // the twelve (tile, digit) columns of the row (lanes 12-15 hold 0)
          v = facc[cg][i];
          v += __shfl_xor(v, 1, 64);
          v += __shfl_xor(v, 2, 64);
          v += __shfl_xor(v, 4, 64);
          v += __shfl_xor(v, 8, 64);
        } else {
          v = facc[cg][i] + __shfl_down(facc[cg][i], 1, 64);
          if constexpr (HD == 3) v += __shfl_down(facc[cg][i], 2, 64);
        }
        if (lead) part[wave][ctok[cg]][kg * 4 + i] += cwgt[cg] * v;
      }
    }
  }
  __syncthreads();
  for (int i = tid; i < T * 16; i += 64 * KS) {
    const int t = i >> 4, r = i & 15;
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < KS; ++w) s += part[w][t][r];
    out[(size_t)t * C + blockIdx.x * 16 + r] = s;
  }
}

// Waves per workgroup: 16 for INT8 (twice the loads in flight per CU of 8
// waves with batches of half the size); 14 for INT4, whose 16-byte loads
// cover two k-steps: R/64 = 224 k-steps then split into 16 per wave and
// expert, two whole batches (Mixtral INT4 decode 0.9 us faster per call; the
// INT8 kernel is 0.4-0.5 us slower with 14)
template <bool I4>
constexpr int down_waves() { return I4 ? 14 : 16; }

template <int NG, bool I4, int HD, bool TE = false>
static void launch_decode_down_ng(const Layout& L, const WsPtr& w, const ExpertPool& ep,
                                  float* out, hipStream_t st) {
  constexpr int KS = down_waves<I4>();
  launch_timed("decode_down", (decode_down_kernel<NG, KS, I4, HD, TE>), dim3(L.C / 16),
               dim3(64 * KS), 0, st, L.C, L.R, L.T, decode_max_active(L), ep, w.dwork, w.hdig,
               w.hexp, out);
}

template <int NG, bool I4>
static void launch_decode_gateup(const Layout& L, const WsPtr& w, const ExpertPool& ep,
                                 hipStream_t st) {
  const int nrb = L.R / kBlk;
  const int max_active = decode_max_active(L);
  if constexpr (I4 && NG == 1) {
    if (L.C <= kXlMaxC) {
      launch_timed("decode_gateup", decode_gateup_xl_kernel, dim3(max_active * nrb), dim3(256), 0, st,
                   L.C, L.R, ep, w.dwork, w.xdig, w.hdig, w.hexp);
      return;
    }
  }
  launch_timed("decode_gateup", (decode_gateup_kernel<NG, I4>), dim3(max_active * nrb),
               dim3(256), 0, st, L.C, L.R, ep, w.dwork, w.xdig, w.hdig, w.hexp);
}

// One token: the 16-row tiles of all active experts split evenly over the
// CUs (W waves per workgroup, about one workgroup per CU), and the down
// kernel reads per-tile exponents.
template <bool I4>
static void launch_decode_ffn_1tok(const Layout& L, const WsPtr& w, const ExpertPool& ep,
                                   float* out, hipStream_t st) {
  const int ntiles = decode_max_active(L) * (L.R / 16);
  const int cus = device_cu_count();
  const int W = std::min(kTileMaxWaves, (ntiles + cus - 1) / cus);
  const int nwg = (ntiles + W - 1) / W;
  launch_timed("decode_gateup", I4 ? decode_gateup_tile_i4_kernel : decode_gateup_tile_kernel,
               dim3(nwg), dim3(64 * W), 0, st, L.C, L.R, W, ntiles, ep, w.dwork, w.xdig, w.hdig,
               w.hexp);
  launch_decode_down_ng<1, I4, 3, true>(L, w, ep, out, st);
}

template <bool I4>
static void launch_decode_ffn(const Layout& L, const WsPtr& w, const ExpertPool& ep, float* out,
                              hipStream_t st) {
  if (L.T == 1 && (!I4 || L.C <= kXlMaxC)) {
    launch_decode_ffn_1tok<I4>(L, w, ep, out, st);
    return;
  }
  // token groups of an expert (each holds at most T tokens): 5 tokens per x
  // operand; H' in three digits for one x group (5 tokens per operand),
  // else in two (8 tokens per operand)
  const int ng = (L.T + kTokPerGroup - 1) / kTokPerGroup;
  switch (ng) {
    case 1: launch_decode_gateup<1, I4>(L, w, ep, st); break;
    case 2: launch_decode_gateup<2, I4>(L, w, ep, st); break;
    case 3: launch_decode_gateup<3, I4>(L, w, ep, st); break;
    default: launch_decode_gateup<4, I4>(L, w, ep, st); break;
  }
  static_assert(MIRA_DECODE_MAX_TOKENS <= 2 * h_tok_per_group(2), "two H' groups cover a decode call");
  if (ng == 1)
    launch_decode_down_ng<1, I4, 3>(L, w, ep, out, st);
  else if (L.T <= h_tok_per_group(2))
    launch_decode_down_ng<1, I4, 2>(L, w, ep, out, st);
  else
    launch_decode_down_ng<2, I4, 2>(L, w, ep, out, st);
}

hipError_t launch_decode(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                         const ExpertPool& ep, float* out, hipStream_t st) {
  (void)x;  // x enters through the fixed-point digits written by decode_prep_kernel
  const int T = L.T;
  if (T == 0) return hipSuccess;
  if (s.flags & MIRA_FLAG_INT4)
    launch_decode_ffn<true>(L, w, ep, out, st);
  else
    launch_decode_ffn<false>(L, w, ep, out, st);
  return hipGetLastError();
}

}  // namespace mira
