// Many-token (prefill) expert FFN over packed experts: grouped GEMMs.
//
// Per expert group g with tokens at positions [off_g, off_g + n_g):
//   gate/up:  H'[pos][r] = sigma_r * silu(sigma_r * (Qg x)_r) * sigma_r * (Qu x)_r   (bf16)
//   down:     Y[pos][c]  = sum_r Qd[c][r] * H'[pos][r]                              (fp32)
//   combine:  out[t] = sum_j w[t,j] * Y[inv[t*k+j]] + sum_s Y[inv[T*k + s*T + t]]
// The int8 weight tiles are widened to bf16 (exact: |q| <= 127) while they are
// staged into LDS, and bf16 MFMA (v_mfma_f32_16x16x32_bf16) accumulates in fp32.
// Tiles (group, n-tile, m-tile) are walked by a persistent grid; the tile
// count is read from the device, so the host never waits for the routing.
#include "device_util.h"
#include "mira_internal.h"

namespace mira {

constexpr int kBK = 64;         // k values per LDS stage
constexpr int kLdsPad = 8;      // bf16 padding per LDS row
constexpr int kLdsRow = kBK + kLdsPad;
constexpr int kGemmThreads = 256;

// Widen 16 int8 values to 16 bf16 (two 16-byte vectors).  int8 -> fp32 is
// exact and an integer of magnitude <= 127 has a zero low half-word in fp32,
// so the bf16 is the upper half-word.
__device__ __forceinline__ void i8x16_to_bf16(v4i q, v4i& lo, v4i& hi) {
  uint32_t o[8];
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const int v = q[w];
    const uint32_t f0 = __float_as_uint((float)(int8_t)(v));
    const uint32_t f1 = __float_as_uint((float)(int8_t)(v >> 8));
    const uint32_t f2 = __float_as_uint((float)(int8_t)(v >> 16));
    const uint32_t f3 = __float_as_uint((float)(v >> 24));
    o[2 * w] = __builtin_amdgcn_perm(f1, f0, 0x07060302u);
    o[2 * w + 1] = __builtin_amdgcn_perm(f3, f2, 0x07060302u);
  }
  lo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  hi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

// BN weight rows (per matrix) x BM tokens per tile; WN x WM per wave.
// DUAL: gate and up matrices with the SwiGLU epilogue writing H' (bf16);
// otherwise the down matrix writing Y (fp32).
template <int BN, int BM, int WN, int WM, bool DUAL>
__global__ __launch_bounds__(kGemmThreads) void prefill_gemm_kernel(
    int C, int R, int G, ExpertPool ep, const int32_t* __restrict__ misc,
    const int32_t* __restrict__ mstart, const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ tokpos, const uint16_t* __restrict__ act,
    uint16_t* __restrict__ hout, float* __restrict__ yout) {
  constexpr int NB = DUAL ? 2 : 1;
  constexpr int WAVES_N = BN / WN, WAVES_M = BM / WM;
  static_assert(WAVES_N * WAVES_M * 64 == kGemmThreads, "wave layout");
  constexpr int NS = WN / 16, MS = WM / 16;
  constexpr int W_CHUNKS = NB * BN * (kBK / 16);  // 16-byte int8 chunks per stage
  constexpr int X_CHUNKS = BM * (kBK / 8);        // 16-byte bf16 chunks per stage
  constexpr int WC_PER_T = (W_CHUNKS + kGemmThreads - 1) / kGemmThreads;
  constexpr int XC_PER_T = (X_CHUNKS + kGemmThreads - 1) / kGemmThreads;

  __shared__ __attribute__((aligned(16))) uint16_t sW[NB * BN][kLdsRow];
  __shared__ __attribute__((aligned(16))) uint16_t sX[BM][kLdsRow];

  const int K = DUAL ? C : R;         // contraction length
  const int N = DUAL ? R : C;         // weight rows per matrix
  const int NT = N / BN;
  const int total = misc[MISC_MTOTAL] * NT;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wn = wave / WAVES_M, wm = wave - wn * WAVES_M;
  const int r16 = lane & 15, kg = lane >> 4;

  for (int tau = blockIdx.x; tau < total; tau += gridDim.x) {
    // group of this tile: the last g with mstart[g]*NT <= tau (tiles of
    // group g occupy [mstart[g]*NT, mstart[g+1]*NT), n-tile major)
    int g = 0;
    {
      int hi = G;
      while (hi - g > 1) {
        const int mid = (g + hi) >> 1;
        if (mstart[mid] * NT <= tau) g = mid;
        else hi = mid;
      }
    }
    const int mt_g = mstart[g + 1] - mstart[g];
    const int local = tau - mstart[g] * NT;
    const int nt = local / mt_g, ml = local - nt * mt_g;
    const int p0 = offsets[g] + ml * BM, p_end = offsets[g + 1];
    const int n0 = nt * BN;
    const int slot = ep.slot_table[g];
    if (slot < 0 || slot >= ep.n_slots) {
      if (tid == 0 && ep.status) atomicOr(ep.status, slot < 0 ? 1 : 2);
      continue;
    }
    const int8_t* blob = ep.pool + (size_t)slot * ep.stride;
    const int8_t* wbase = blob + (DUAL ? 0 : (size_t)2 * R * C);

    // per-thread global sources of this tile.  Weight chunks walk whole
    // 1 KB tiles of the packed layout (16 rows x 64 k, run g*16+i = row i,
    // k 16g..16g+15), so consecutive lanes read consecutive 16 bytes.
    const int8_t* wsrc[WC_PER_T];
    int wdst[WC_PER_T];
#pragma unroll
    for (int i = 0; i < WC_PER_T; ++i) {
      const int ch = tid + i * kGemmThreads;
      const int tl = ch >> 6, run = ch & 63;                    // tile of the stage, run in it
      const int mat = tl / (BN / 16), rt = tl - mat * (BN / 16);
      const int row = mat * BN + rt * 16 + (run & 15), part = run >> 4;
      wsrc[i] = wbase + (size_t)mat * R * C + (size_t)(n0 / 16 + rt) * (K / 64) * 1024 + run * 16;
      wdst[i] = ch < W_CHUNKS ? row * kLdsRow + part * 16 : -1;
    }
    const uint16_t* xsrc[XC_PER_T];
    int xdst[XC_PER_T];
    bool xok[XC_PER_T];
#pragma unroll
    for (int i = 0; i < XC_PER_T; ++i) {
      const int ch = tid + i * kGemmThreads;
      const int row = ch / (kBK / 8), part = ch - row * (kBK / 8);
      const int pos = p0 + row;
      xok[i] = ch < X_CHUNKS && pos < p_end;
      const int src_row = xok[i] ? (DUAL ? tokpos[pos] : pos) : 0;
      xsrc[i] = act + (size_t)src_row * K + part * 8;
      xdst[i] = ch < X_CHUNKS ? row * kLdsRow + part * 8 : -1;
    }

    v4f acc[NB][NS][MS];
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int ns = 0; ns < NS; ++ns)
#pragma unroll
        for (int ms = 0; ms < MS; ++ms) acc[b][ns][ms] = v4f{0.f, 0.f, 0.f, 0.f};

    v4i wreg[WC_PER_T], xreg[XC_PER_T];
    auto gload = [&](int k0) {
#pragma unroll
      for (int i = 0; i < WC_PER_T; ++i)
        wreg[i] = wdst[i] >= 0 ? ld16_stream(wsrc[i] + (size_t)(k0 >> 6) * 1024) : zero16();
#pragma unroll
      for (int i = 0; i < XC_PER_T; ++i) xreg[i] = xok[i] ? ld16(xsrc[i] + k0) : zero16();
    };
    auto lstore = [&]() {
#pragma unroll
      for (int i = 0; i < WC_PER_T; ++i) {
        if (wdst[i] < 0) continue;
        v4i lo, hi;
        i8x16_to_bf16(wreg[i], lo, hi);
        *(v4i*)(&sW[0][0] + wdst[i]) = lo;
        *(v4i*)(&sW[0][0] + wdst[i] + 8) = hi;
      }
#pragma unroll
      for (int i = 0; i < XC_PER_T; ++i)
        if (xdst[i] >= 0) *(v4i*)(&sX[0][0] + xdst[i]) = xreg[i];
    };

    gload(0);
    for (int k0 = 0; k0 < K; k0 += kBK) {
      __syncthreads();  // previous stage fully consumed
      lstore();
      __syncthreads();
      if (k0 + kBK < K) gload(k0 + kBK);
#pragma unroll
      for (int kk = 0; kk < kBK; kk += 32) {
        v4i af[NB][NS], bf[MS];
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int ns = 0; ns < NS; ++ns)
            af[b][ns] = *(const v4i*)(&sW[b * BN + wn * WN + ns * 16 + r16][kk + kg * 8]);
#pragma unroll
        for (int ms = 0; ms < MS; ++ms)
          bf[ms] = *(const v4i*)(&sX[wm * WM + ms * 16 + r16][kk + kg * 8]);
#pragma unroll
        for (int b = 0; b < NB; ++b)
#pragma unroll
          for (int ns = 0; ns < NS; ++ns)
#pragma unroll
            for (int ms = 0; ms < MS; ++ms) acc[b][ns][ms] = mfma_bf16(af[b][ns], bf[ms], acc[b][ns][ms]);
      }
    }

    // epilogue: acc[b][ns][ms][i] = row n0 + wn*WN + ns*16 + kg*4 + i, token p0 + wm*WM + ms*16 + r16
#pragma unroll
    for (int ns = 0; ns < NS; ++ns) {
      const int rr = n0 + wn * WN + ns * 16 + kg * 4;
      float sg[4];
      if (DUAL) {
        const uint16_t* sig = (const uint16_t*)(blob + (size_t)3 * R * C);
#pragma unroll
        for (int i = 0; i < 4; ++i) sg[i] = bf16_to_f32(sig[rr + i]);
      }
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int pos = p0 + wm * WM + ms * 16 + r16;
        if (pos >= p_end) continue;
        if (DUAL) {
          uint32_t hb[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float gv = sg[i] * acc[0][ns][ms][i];
            const float uv = sg[i] * acc[NB - 1][ns][ms][i];
            const float h = sg[i] * (gv / (1.f + expf(-gv)) * uv);
            hb[i] = f32_to_bf16_rne(h);
          }
          uint2 pk;
          pk.x = hb[0] | (hb[1] << 16);
          pk.y = hb[2] | (hb[3] << 16);
          *(uint2*)(hout + (size_t)pos * R + rr) = pk;
        } else {
          *(v4f*)(yout + (size_t)pos * C + rr) = acc[0][ns][ms];
        }
      }
    }
  }
}

// out[t][c] = sum_j w[t][j] * Y[inv[t*k+j]][c] + sum_s Y[inv[T*k + s*T + t]][c]
__global__ __launch_bounds__(256) void combine_kernel(int T, int C, int k, int S,
                                                      const int32_t* __restrict__ inv,
                                                      const float* __restrict__ wts,
                                                      const float* __restrict__ y,
                                                      float* __restrict__ out) {
  const int t = blockIdx.y;
  const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (c >= C) return;
  v4f s = {0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < k; ++j) {
    const float w = wts[(size_t)t * k + j];
    const v4f v = *(const v4f*)(y + (size_t)inv[(size_t)t * k + j] * C + c);
    s += w * v;
  }
  for (int sh = 0; sh < S; ++sh) {
    const v4f v = *(const v4f*)(y + (size_t)inv[(size_t)T * k + (size_t)sh * T + t] * C + c);
    s += v;
  }
  *(v4f*)(out + (size_t)t * C + c) = s;
}

__global__ __launch_bounds__(256) void f32_to_bf16_kernel(const float* __restrict__ x,
                                                          uint16_t* __restrict__ y, size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
    y[i] = f32_to_bf16_rne(x[i]);
}

// tile shapes
constexpr int kGU_BN = 64, kGU_WN = 32, kGU_WM = 32;
constexpr int kDN_BN = 64, kDN_WN = 32, kDN_WM = 32;

template <typename Kern>
static int persistent_grid(Kern k, int& occ_cache, int max_tiles) {
  if (occ_cache <= 0) {
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, k, kGemmThreads, 0) != hipSuccess ||
        occ < 1)
      occ = 1;
    occ_cache = occ;
  }
  const long cap = (long)device_cu_count() * occ_cache;
  return (int)(max_tiles < cap ? max_tiles : cap);
}

hipError_t launch_prefill(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                          const ExpertPool& ep, float* out, hipStream_t st) {
  const int T = L.T;
  if (T == 0) return hipSuccess;
  const uint16_t* xb = (const uint16_t*)x;
  if (s.act_dtype == MIRA_F32) {
    const size_t n = (size_t)T * L.C;
    const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
    prof_begin("prefill_cvt", st);
    hipLaunchKernelGGL(f32_to_bf16_kernel, dim3(blocks), dim3(256), 0, st, (const float*)x,
                       w.xb16, n);
    prof_end("prefill_cvt", st);
    xb = w.xb16;
  }
  {
    auto kern = prefill_gemm_kernel<kGU_BN, kPrefBM, kGU_WN, kGU_WM, true>;
    static int occ = 0;
    const int grid = persistent_grid(kern, occ, L.mt_max * (L.R / kGU_BN));
    prof_begin("prefill_gateup", st);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kGemmThreads), 0, st, L.C, L.R, L.G, ep, w.misc,
                       w.mstart, w.offsets, w.tokpos, xb, w.hbuf, (float*)nullptr);
    prof_end("prefill_gateup", st);
  }
  {
    auto kern = prefill_gemm_kernel<kDN_BN, kPrefBM, kDN_WN, kDN_WM, false>;
    static int occ = 0;
    const int grid = persistent_grid(kern, occ, L.mt_max * (L.C / kDN_BN));
    prof_begin("prefill_down", st);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(kGemmThreads), 0, st, L.C, L.R, L.G, ep, w.misc,
                       w.mstart, w.offsets, w.tokpos, (const uint16_t*)w.hbuf, (uint16_t*)nullptr,
                       w.ybuf);
    prof_end("prefill_down", st);
  }
  {
    dim3 grid((L.C / 4 + 255) / 256, T);
    prof_begin("prefill_combine", st);
    hipLaunchKernelGGL(combine_kernel, grid, dim3(256), 0, st, T, L.C, L.k, L.S, w.inv, w.wts,
                       w.ybuf, out);
    prof_end("prefill_combine", st);
  }
  return hipGetLastError();
}

}  // namespace mira
