// Device body of the small-batch (decode) gate/up kernel: one block of 64
// expert rows for the tokens of one expert group.
//
// The paper fuses INT8 dequantization into the expert FFN (sections IV-A and
// IV-F).  Because the scale sigma_r is shared by gate row r, up row r and down
// column r (section IV-B), it factors out of every dot product:
//   G = sigma (.) (Qg x),  U = sigma (.) (Qu x),  H' = sigma (.) silu(G) (.) U.
// The packed int8 bytes go unchanged to the int8 matrix cores
// (v_mfma_i32_16x16x64_i8); the activation side is a fixed-point integer
// split into three signed base-256 digits, each digit one int8 operand
// column, so products and sums are exact int32.  Five tokens (15 digit
// columns) fit one 16-column operand.
#pragma once

#include "device_util.h"
#include "int4_format.h"
#include "mira_internal.h"

namespace mira {

// Combine the three digit columns held by lanes j, j+1, j+2 (j = 3m) into
// the exact integer dot product.
__device__ __forceinline__ float combine_digits_i(int s0) {
  const int s1 = __shfl_down(s0, 1, 64);
  const int s2 = __shfl_down(s0, 2, 64);
  const long long v = (long long)s2 * 65536 + (long long)s1 * 256 + (long long)s0;
  return (float)v;
}

// k-steps per load batch; fewer when many token groups need registers
__host__ __device__ constexpr int dec_unroll(int ng) { return ng == 1 ? 16 : ng == 2 ? 8 : 4; }

// H' of one 64-row block as fixed-point digits with one exponent per token
// and block: bmax holds each wave's per-token maxima of |hv|; lane (kg, r16)
// holds rows rb*64 + wave*16 + kg*4 + i of token column r16 (lead lanes).
// With HD = 3 digits H' has kFixBits bits against the block maximum, with
// HD = 2 kHFixBits2; balanced base-256 digits hdig[(pos*HD + d)*R + r] and
// the exponent hexp[pos*(R/64) + rb].
template <int NG>
__device__ __forceinline__ void write_h_digits(int R, int rb, int off, bool lead,
                                               const bool (&bv)[NG], const float (&hv)[NG][4],
                                               int8_t* __restrict__ hdig,
                                               int32_t* __restrict__ hexp,
                                               float (*bmax)[NG * kTokPerGroup]) {
  constexpr int HD = h_digits(NG);
  const int nrb = R / kBlk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int m = r16 / 3;
  const int rbase = rb * kBlk + wave * 16 + kg * 4;
  __syncthreads();
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    if (!(lead && bv[cg])) continue;
    const int ti = cg * kTokPerGroup + m;
    const float mx = fmaxf(fmaxf(bmax[0][ti], bmax[1][ti]), fmaxf(bmax[2][ti], bmax[3][ti]));
    const int Eh = (HD == 3 ? kFixBits : kHFixBits2) - exp_bound(mx);
    uint32_t w0 = 0, w1 = 0, w2 = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // |hv| <= mx < 2^exp_bound(mx): |v| <= 2^22 (2^14), so the top digit
      // stays within [-64, 64]
      const int v = (int)rintf(ldexpf(hv[cg][i], Eh));
      int d0, d1, d2;
      if constexpr (HD == 3) {
        split_digits(v, d0, d1, d2);
      } else {
        d0 = (int)(int8_t)(v & 0xFF);
        d1 = (v - d0) >> 8;
        d2 = 0;
      }
      w0 |= (uint32_t)(d0 & 0xFF) << (8 * i);
      w1 |= (uint32_t)(d1 & 0xFF) << (8 * i);
      w2 |= (uint32_t)(d2 & 0xFF) << (8 * i);
    }
    const size_t pos = (size_t)off + ti;
    int8_t* hp = hdig + pos * HD * R + rbase;
    *(uint32_t*)(hp) = w0;
    *(uint32_t*)(hp + R) = w1;
    if constexpr (HD == 3) *(uint32_t*)(hp + 2 * (size_t)R) = w2;
    if (wave == 0 && kg == 0) hexp[pos * nrb + rb] = Eh;
  }
}

// Gate and up sums of one 16-row tile (rows 16*rtile .. +15) for the tokens
// of one expert group, by one wave.  Token column r16 of operand group cg is
// token cg*5 + r16/3, digit r16%3; bv[cg] says whether that column holds a
// token.  load_b(cg, ks) returns this lane's 16 digit bytes of k-step ks
// (k = 64*ks + 16*(lane/16) .. +15).  On return accg/accu hold the int32
// digit sums of rows 16*rtile + 4*(lane/16) + i (i < 4) for column r16, and
// sg those rows' scales sigma_r.
template <int NG, typename LoadB>
__device__ __forceinline__ void gateup_tile_stream(int C, int R, int rtile,
                                                   const int8_t* __restrict__ blob,
                                                   const bool (&bv)[NG], LoadB load_b,
                                                   v4i (&accg)[NG], v4i (&accu)[NG],
                                                   float (&sg)[4]) {
  const int lane = threadIdx.x & 63, kg = lane >> 4;
  // the tile: 1 KB per k-step, lane l at byte 16*l
  const int8_t* gp = blob + (size_t)rtile * (C / 64) * 1024 + lane * 16;
  const int8_t* up = gp + (size_t)R * C;
  // the four bf16 scales of this lane's rows are one 8-byte load, issued
  // ahead of the stream so that it returns with the first batch instead of
  // costing a round trip at the end
  const int rbase = rtile * 16 + kg * 4;
  const uint2 sraw = *(const uint2*)(blob + (size_t)3 * R * C + (size_t)rbase * 2);

#pragma unroll
  for (int cg = 0; cg < NG; ++cg) accg[cg] = accu[cg] = zero16();

  constexpr int kDecUnroll = dec_unroll(NG);
  const int nks = C / 64;
  struct Batch {
    v4i ag[kDecUnroll], au[kDecUnroll], b[kDecUnroll][NG];
  };
  auto issue = [&](Batch& bt, int ks0) {
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u) {
      const int ks = ks0 + u;
      const bool in = ks < nks;
      bt.ag[u] = in ? ld16_stream(gp + ks * 1024) : zero16();
      bt.au[u] = in ? ld16_stream(up + ks * 1024) : zero16();
#pragma unroll
      for (int cg = 0; cg < NG; ++cg) bt.b[u][cg] = (in && bv[cg]) ? load_b(cg, ks) : zero16();
    }
  };
  auto consume = [&](const Batch& bt) {
#pragma unroll
    for (int u = 0; u < kDecUnroll; ++u)
#pragma unroll
      for (int cg = 0; cg < NG; ++cg) {
        accg[cg] = mfma_i8(bt.ag[u], bt.b[u][cg], accg[cg]);
        accu[cg] = mfma_i8(bt.au[u], bt.b[u][cg], accu[cg]);
      }
  };
  // one batch per iteration, issued whole and consumed in order: no load
  // result is carried around the loop, so the waits count down within the
  // batch instead of draining at the back edge
  for (int ks = 0; ks < nks; ks += kDecUnroll) {
    Batch bt;
    issue(bt, ks);
    consume(bt);
  }

  sg[0] = __uint_as_float(sraw.x << 16);
  sg[1] = __uint_as_float(sraw.x & 0xffff0000u);
  sg[2] = __uint_as_float(sraw.y << 16);
  sg[3] = __uint_as_float(sraw.y & 0xffff0000u);
}

// H' of one row from its gate and up digit sums: with xs = 2^-E of the
// token's fixed point, G = sigma*xs*gsum, U = sigma*xs*usum and
// H' = sigma * silu(G) * U (the shared scale of down column r).
__device__ __forceinline__ float swiglu_h(int gsum_digits, int usum_digits, float xs, float sig) {
  const float gv = combine_digits_i(gsum_digits) * xs * sig;
  const float uv = combine_digits_i(usum_digits) * xs * sig;
  return sig * (gv / (1.f + expf(-gv)) * uv);
}

// Gate/up + SwiGLU of one block of 64 expert rows (rb) for the tokens of one
// expert group, by a workgroup of 4 waves (wave w owns rows rb*64 + 16w ..
// +15, streamed by gateup_tile_stream); xev[cg] is the token's fixed-point
// exponent.  Writes H' of the group's positions off .. off+n-1 as per-block
// fixed-point digits (write_h_digits).
template <int NG, typename LoadB>
__device__ __forceinline__ void gateup_block(int C, int R, int rb, const int8_t* __restrict__ blob,
                                             int off, const bool (&bv)[NG], const int (&xev)[NG],
                                             LoadB load_b, int8_t* __restrict__ hdig,
                                             int32_t* __restrict__ hexp,
                                             float (*bmax)[NG * kTokPerGroup]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int m = r16 / 3, d = r16 - 3 * m;
  v4i accg[NG], accu[NG];
  float sg[4];
  gateup_tile_stream<NG>(C, R, rb * (kBlk / 16) + wave, blob, bv, load_b, accg, accu, sg);

  const bool lead = d == 0;
  float hv[NG][4];
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    const float xs = bv[cg] ? ldexpf(1.f, -xev[cg]) : 0.f;
    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float h = swiglu_h(accg[cg][i], accu[cg][i], xs, sg[i]);
      hv[cg][i] = (lead && bv[cg]) ? h : 0.f;
      mx = fmaxf(mx, fabsf(hv[cg][i]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (kg == 0 && lead && r16 < 3 * kTokPerGroup) bmax[wave][cg * kTokPerGroup + m] = mx;
  }
  write_h_digits<NG>(R, rb, off, lead, bv, hv, hdig, hexp, bmax);
}

// One-token groups: writes H' of one 16-row tile (rows 16*rt .. +15) with
// the tile's own exponent: three balanced base-256 digits
// hdig[(pos*3 + d)*R + r] with kFixBits bits against the tile maximum and
// hexp[pos*(R/16) + rt].  Lane (r16, kg) with lead set holds the token's
// rows 16*rt + 4*kg + i in hv (hv = 0 elsewhere); the lead lanes are r16 ==
// 0.  (The down kernel gives each (tile, digit) pair of a k-step its own
// operand column, so the four tiles of a k-step need no common exponent.)
__device__ __forceinline__ void write_h_tile_1tok(int R, int rt, int pos, bool lead,
                                                  const float (&hv)[4], int8_t* __restrict__ hdig,
                                                  int32_t* __restrict__ hexp) {
  const int lane = threadIdx.x & 63, kg = lane >> 4;
  float mx = 0.f;
#pragma unroll
  for (int i = 0; i < 4; ++i) mx = fmaxf(mx, fabsf(hv[i]));
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  if (!lead) return;
  const int Eh = kFixBits - exp_bound(mx);
  uint32_t w0 = 0, w1 = 0, w2 = 0;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    // |hv| <= mx < 2^exp_bound(mx): |v| <= 2^22, so the top digit stays
    // within [-64, 64]
    int d0, d1, d2;
    split_digits((int)rintf(ldexpf(hv[i], Eh)), d0, d1, d2);
    w0 |= (uint32_t)(d0 & 0xFF) << (8 * i);
    w1 |= (uint32_t)(d1 & 0xFF) << (8 * i);
    w2 |= (uint32_t)(d2 & 0xFF) << (8 * i);
  }
  int8_t* hp = hdig + (size_t)pos * 3 * R + rt * 16 + kg * 4;
  *(uint32_t*)(hp) = w0;
  *(uint32_t*)(hp + R) = w1;
  *(uint32_t*)(hp + 2 * (size_t)R) = w2;
  if (kg == 0) hexp[(size_t)pos * (R / 16) + rt] = Eh;
}

// One-token INT8 tile: H' = sigma (.) silu(G) (.) U from the gate and up
// digit sums (lane (r16, kg) holds rows 16*rt + 4*kg + i of digit column
// r16), written by write_h_tile_1tok.  sg: the rows' scales sigma_r; xe: the
// token's fixed-point exponent.
__device__ __forceinline__ void h_tile_1tok(int R, int rt, int pos, bool bv, int xe, v4i accg,
                                            v4i accu, const float (&sg)[4],
                                            int8_t* __restrict__ hdig,
                                            int32_t* __restrict__ hexp) {
  const int r16 = threadIdx.x & 15;
  const bool lead = bv && r16 == 0;
  const float xs = bv ? ldexpf(1.f, -xe) : 0.f;
  float hv[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float h = swiglu_h(accg[i], accu[i], xs, sg[i]);
    hv[i] = lead ? h : 0.f;
  }
  write_h_tile_1tok(R, rt, pos, lead, hv, hdig, hexp);
}

// ---- INT4 variant (MIRA_FLAG_INT4) -----------------------------------------
// 8 bytes of one 16-column run -> the int8 operand of those 16 columns, each
// as 16*q: the run order puts columns 0-3 (8-11) in the high nibbles and
// columns 4-7 (12-15) in the low nibbles of the first (second) dword.
__device__ __forceinline__ v4i i4_operand(uint2 p) {
  return v4i{(int)(p.x & 0xF0F0F0F0u), (int)((p.x << 4) & 0xF0F0F0F0u),
             (int)(p.y & 0xF0F0F0F0u), (int)((p.y << 4) & 0xF0F0F0F0u)};
}

typedef unsigned int v2u __attribute__((ext_vector_type(2)));

__device__ __forceinline__ uint2 ld8_stream(const void* p) {
  const v2u v = __builtin_nontemporal_load((const v2u*)p);
  return uint2{v[0], v[1]};
}

// four fp16 scales (rows 4*kg .. 4*kg+3 of a tile) to fp32
__device__ __forceinline__ void i4_scales(uint2 p, float (&s)[4]) {
  s[0] = (float)__builtin_bit_cast(_Float16, (uint16_t)(p.x & 0xFFFFu));
  s[1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(p.x >> 16));
  s[2] = (float)__builtin_bit_cast(_Float16, (uint16_t)(p.y & 0xFFFFu));
  s[3] = (float)__builtin_bit_cast(_Float16, (uint16_t)(p.y >> 16));
}

// Float version of combine_digits_i for per-group scaled sums.
__device__ __forceinline__ float combine_digits_f(float s0) {
  const float s1 = __shfl_down(s0, 1, 64);
  const float s2 = __shfl_down(s0, 2, 64);
  return s2 * 65536.f + s1 * 256.f + s0;
}

// Gate and up sums of one 16-row INT4 tile (rows 16*rtile .. +15) by one
// wave, with the operands of gateup_tile_stream.  Each k-step is one
// 64-column group: the MFMA sums of that group are scaled by the group's
// fp16 scale (per row) and accumulated in fp32 (accg/accu, still per digit
// column).  U k-steps per load batch; with B_AT_USE the activation digits
// are read (from LDS) right before their MFMAs instead of travelling with
// the weight loads, so a batch holds only weight registers.
template <int NG, int U, bool B_AT_USE, typename LoadB>
__device__ __forceinline__ void gateup_tile_stream_i4(int C, int R, int rtile,
                                                      const uint8_t* __restrict__ blob,
                                                      const bool (&bv)[NG], LoadB load_b,
                                                      float (&accg)[NG][4], float (&accu)[NG][4]) {
  const int lane = threadIdx.x & 63, kg = lane >> 4;
  const int nks = C / 64, npair = C / 128;
  // the tile-row: nibble tiles of two groups (lane l's 16 bytes at 16*l)
  // and the 32-byte scale blocks of its groups
  const size_t mbytes = i4_matrix_bytes(R, C), nbytes = i4_nib_bytes(R, C);
  const uint8_t* gq = blob + (size_t)rtile * npair * kI4PairTile + lane * 16;
  const uint8_t* uq = gq + mbytes;
  const uint8_t* gs = blob + nbytes + (size_t)rtile * nks * 32 + lane * 8;
  const uint8_t* us = gs + mbytes;

#pragma unroll
  for (int cg = 0; cg < NG; ++cg)
#pragma unroll
    for (int i = 0; i < 4; ++i) accg[cg][i] = accu[cg][i] = 0.f;

  static_assert(U % 2 == 0 && U <= 16, "a batch covers whole tiles and one scale run");
  constexpr int kDecUnroll = U;
  struct Batch {
    v4i qg[U / 2], qu[U / 2];  // two k-steps per 16-byte load
    uint2 sg, su;              // lane l: group ks0 + l/4, rows 4*(l%4) .. +3
    v4i b[B_AT_USE ? 1 : U][NG];
    int ks0;
  };
  auto issue = [&](Batch& bt, int ks0) {
#pragma unroll
    for (int p = 0; p < U / 2; ++p) {
      const int pair = ks0 / 2 + p;
      const bool in = pair < npair;
      bt.qg[p] = in ? ld16_stream(gq + (size_t)pair * kI4PairTile) : zero16();
      bt.qu[p] = in ? ld16_stream(uq + (size_t)pair * kI4PairTile) : zero16();
    }
    const bool sin = (lane >> 2) < U && ks0 + (lane >> 2) < nks;
    bt.sg = sin ? ld8_stream(gs + (size_t)ks0 * 32) : uint2{0, 0};
    bt.su = sin ? ld8_stream(us + (size_t)ks0 * 32) : uint2{0, 0};
    if constexpr (!B_AT_USE) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const bool in = ks0 + u < nks;
#pragma unroll
        for (int cg = 0; cg < NG; ++cg) bt.b[u][cg] = (in && bv[cg]) ? load_b(cg, ks0 + u) : zero16();
      }
    }
    bt.ks0 = ks0;
  };
  auto consume = [&](const Batch& bt) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const v4i g2 = bt.qg[u / 2], u2 = bt.qu[u / 2];
      const v4i ag = (u & 1) ? i4_operand(uint2{(uint32_t)g2[2], (uint32_t)g2[3]})
                             : i4_operand(uint2{(uint32_t)g2[0], (uint32_t)g2[1]});
      const v4i au = (u & 1) ? i4_operand(uint2{(uint32_t)u2[2], (uint32_t)u2[3]})
                             : i4_operand(uint2{(uint32_t)u2[0], (uint32_t)u2[1]});
      // this lane's four row scales of group ks0 + u sit in lane 4u + kg
      float sgv[4], suv[4];
      i4_scales(uint2{(uint32_t)__shfl((int)bt.sg.x, 4 * u + kg, 64),
                      (uint32_t)__shfl((int)bt.sg.y, 4 * u + kg, 64)}, sgv);
      i4_scales(uint2{(uint32_t)__shfl((int)bt.su.x, 4 * u + kg, 64),
                      (uint32_t)__shfl((int)bt.su.y, 4 * u + kg, 64)}, suv);
#pragma unroll
      for (int cg = 0; cg < NG; ++cg) {
        v4i bo;
        if constexpr (B_AT_USE)
          bo = bt.ks0 + u < nks ? load_b(cg, bt.ks0 + u) : zero16();
        else
          bo = bt.b[u][cg];
        const v4i rg = mfma_i8(ag, bo, zero16());
        const v4i ru = mfma_i8(au, bo, zero16());
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          accg[cg][i] = fmaf((float)rg[i], sgv[i], accg[cg][i]);
          accu[cg][i] = fmaf((float)ru[i], suv[i], accu[cg][i]);
        }
      }
    }
  };
  // one batch per iteration, issued whole and consumed in order: no load
  // result is carried around the loop, so the waits count down within the
  // batch instead of draining at the back edge
  for (int ks = 0; ks < nks; ks += kDecUnroll) {
    Batch bt;
    issue(bt, ks);
    consume(bt);
  }
}

// Gate/up + SwiGLU of one block of 64 expert rows for INT4 experts: the same
// work split, operands and output as gateup_block; each wave streams its
// tile with gateup_tile_stream_i4, and H' = silu(G) (.) U (no shared scale to
// fold).
template <int NG, int U, bool B_AT_USE, typename LoadB>
__device__ __forceinline__ void gateup_block_i4(int C, int R, int rb, const uint8_t* __restrict__ blob,
                                                int off, const bool (&bv)[NG], const int (&xev)[NG],
                                                LoadB load_b, int8_t* __restrict__ hdig,
                                                int32_t* __restrict__ hexp,
                                                float (*bmax)[NG * kTokPerGroup]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int m = r16 / 3, d = r16 - 3 * m;
  float accg[NG][4], accu[NG][4];
  gateup_tile_stream_i4<NG, U, B_AT_USE>(C, R, rb * (kBlk / 16) + wave, blob, bv, load_b, accg, accu);

  const bool lead = d == 0;
  float hv[NG][4];
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    // 2^-E of the token's fixed point, and 1/16 for the nibble operand (16*q)
    const float xs = bv[cg] ? ldexpf(1.f, -xev[cg] - 4) : 0.f;
    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float gv = combine_digits_f(accg[cg][i]) * xs;
      const float uv = combine_digits_f(accu[cg][i]) * xs;
      const float h = gv / (1.f + expf(-gv)) * uv;
      hv[cg][i] = (lead && bv[cg]) ? h : 0.f;
      mx = fmaxf(mx, fabsf(hv[cg][i]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (kg == 0 && lead && r16 < 3 * kTokPerGroup) bmax[wave][cg * kTokPerGroup + m] = mx;
  }
  write_h_digits<NG>(R, rb, off, lead, bv, hv, hdig, hexp, bmax);
}

}  // namespace mira
