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
__host__ __device__ constexpr int dec_unroll(int ng) { return ng <= 2 ? 4 : 2; }

// Gate/up + SwiGLU of one block of 64 expert rows (rb) for the tokens of one
// expert group, by a workgroup of 4 waves (wave w owns rows rb*64 + 16w ..
// +15).  Token column r16 of operand group cg is token cg*5 + r16/3, digit
// r16%3; bv[cg] says whether that column holds a token and xev[cg] is the
// token's fixed-point exponent.  load_b(cg, ks) returns this lane's 16 digit
// bytes of k-step ks (k = 64*ks + 16*(lane/16) .. +15).  Writes H' of the
// group's positions off .. off+n-1 as per-block fixed-point digits:
// hdig[(pos*3 + d)*R + r], hexp[pos*(R/64) + rb].
template <int NG, typename LoadB>
__device__ __forceinline__ void gateup_block(int C, int R, int rb, const int8_t* __restrict__ blob,
                                             int off, const bool (&bv)[NG], const int (&xev)[NG],
                                             LoadB load_b, int8_t* __restrict__ hdig,
                                             int32_t* __restrict__ hexp,
                                             float (*bmax)[NG * kTokPerGroup]) {
  const int nrb = R / kBlk;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int r16 = lane & 15, kg = lane >> 4;
  const int m = r16 / 3, d = r16 - 3 * m;
  // this wave's 16-row tile: 1 KB per k-step, lane l at byte 16*l
  const int rtile = rb * (kBlk / 16) + wave;
  const int8_t* gp = blob + (size_t)rtile * (C / 64) * 1024 + lane * 16;
  const int8_t* up = gp + (size_t)R * C;

  v4i accg[NG], accu[NG];
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) accg[cg] = accu[cg] = zero16();

  // two batches of U k-steps in flight: issue one, consume the other
  constexpr int kDecUnroll = dec_unroll(NG);
  const int nks = C / 64;
  struct Batch {
    v4i ag[kDecUnroll], au[kDecUnroll], b[kDecUnroll][NG];
  } b0, b1;
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
  issue(b0, 0);
  for (int ks = 0; ks < nks; ks += 2 * kDecUnroll) {
    issue(b1, ks + kDecUnroll);
    consume(b0);
    issue(b0, ks + 2 * kDecUnroll);
    consume(b1);
  }

  // epilogue: rows rbase+i (i < 4) for token column r16
  const int rbase = rb * kBlk + wave * 16 + kg * 4;
  const uint16_t* sig = (const uint16_t*)(blob + (size_t)3 * R * C);
  float sg[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) sg[i] = bf16_to_f32(sig[rbase + i]);
  const bool lead = d == 0;
  float hv[NG][4];
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    const float xs = bv[cg] ? ldexpf(1.f, -xev[cg]) : 0.f;
    float mx = 0.f;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const float gsum = combine_digits_i(accg[cg][i]);
      const float usum = combine_digits_i(accu[cg][i]);
      const float gv = gsum * xs * sg[i];
      const float uv = usum * xs * sg[i];
      const float h = gv / (1.f + expf(-gv)) * uv;
      hv[cg][i] = (lead && bv[cg]) ? sg[i] * h : 0.f;
      mx = fmaxf(mx, fabsf(hv[cg][i]));
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    if (kg == 0 && lead && r16 < 3 * kTokPerGroup) bmax[wave][cg * kTokPerGroup + m] = mx;
  }
  __syncthreads();
#pragma unroll
  for (int cg = 0; cg < NG; ++cg) {
    if (!(lead && bv[cg])) continue;
    const int ti = cg * kTokPerGroup + m;
    const float mx = fmaxf(fmaxf(bmax[0][ti], bmax[1][ti]), fmaxf(bmax[2][ti], bmax[3][ti]));
    const int Eh = kFixBits - exp_bound(mx);
    uint32_t w0 = 0, w1 = 0, w2 = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int v = (int)rintf(ldexpf(hv[cg][i], Eh));
      int d0, d1, d2;
      split_digits(v, d0, d1, d2);
      w0 |= (uint32_t)(d0 & 0xFF) << (8 * i);
      w1 |= (uint32_t)(d1 & 0xFF) << (8 * i);
      w2 |= (uint32_t)(d2 & 0xFF) << (8 * i);
    }
    const size_t pos = (size_t)off + ti;
    int8_t* hp = hdig + pos * kDigits * R + rbase;
    *(uint32_t*)(hp) = w0;
    *(uint32_t*)(hp + R) = w1;
    *(uint32_t*)(hp + 2 * (size_t)R) = w2;
    if (wave == 0 && kg == 0) hexp[pos * nrb + rb] = Eh;
  }
}

}  // namespace mira
