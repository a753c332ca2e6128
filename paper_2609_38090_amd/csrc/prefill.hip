// Many-token (prefill) expert FFN over packed experts: grouped GEMMs.
//
// Per expert group g with tokens at positions [off_g, off_g + n_g):
//   gate/up:  H'[pos][r] = sigma_r * silu(sigma_r * (Qg x)_r) * sigma_r * (Qu x)_r   (bf16)
//   down:     Y[s][pos][c] = sum over the s-th k-chunk of r of Qd[c][r] * H'[pos][r]   (fp32)
//   combine:  out[t] = sum_j w[t,j] * sum_s Y[s][inv[t*k+j]] + shared experts
// A workgroup owns a tile of 512 weight rows (gate/up: 256 of each) by 128
// tokens; its 4 waves split the weight rows, so every wave covers the same
// tokens and all of them skip the 16-token subtiles past the group's end.
// Packed int8 tiles go to LDS as they are (a ring of three stages, loads two
// stages ahead) and each wave widens its own 16x32 operand fragments to bf16
// (exact: |q| <= 127) right before v_mfma_f32_16x16x32_bf16, which
// accumulates in fp32.  Tiles (group, n-tile, k-chunk, m-tile) are walked by
// a persistent grid whose tile count is read from the device, so the host
// never waits for the routing; consecutive tiles share weights and land on
// the same XCD (its L2).
#include <mutex>
#include <type_traits>

#include "device_util.h"
#include "mira_internal.h"

namespace mira {

constexpr int kGemmThreads = 256;                 // 4 waves, one per SIMD
constexpr int kWaveTiles = 8;                     // 16-row packed tiles per wave
constexpr int kTileRows = 4 * kWaveTiles * 16;    // 512 weight rows per workgroup tile
constexpr int kNStage = 3;                        // LDS ring: two stages in flight
constexpr int kWStage = kTileRows * 64;           // 32 KB of packed tiles per stage
constexpr int kXStage = kPrefBM * 64 * 2;         // 16 KB of tokens (128 x 64 bf16)
constexpr int kStageBytes = kWStage + kXStage;    // 48 KB
constexpr int kDmaPerStage = 12;                  // loads per wave and stage: 8 tiles, 4 row groups
static_assert(kPrefBM == 128, "the token stage holds 128 rows");
static_assert(kNStage * kStageBytes <= 160 * 1024, "LDS ring exceeds 160 KB");

// 16 int8 -> two groups of 8 bf16.  int8 -> fp32 is exact and an integer of
// magnitude <= 127 has a zero low half-word in fp32, so its bf16 is the
// upper half-word.
__device__ __forceinline__ void i8x16_to_bf16(v4i q, v4i& lo, v4i& hi) {
  uint32_t o[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = q[j];
    const uint32_t f0 = __float_as_uint((float)(int8_t)(v));
    const uint32_t f1 = __float_as_uint((float)(int8_t)(v >> 8));
    const uint32_t f2 = __float_as_uint((float)(int8_t)(v >> 16));
    const uint32_t f3 = __float_as_uint((float)(v >> 24));
    o[2 * j] = __builtin_amdgcn_perm(f1, f0, 0x07060302u);
    o[2 * j + 1] = __builtin_amdgcn_perm(f3, f2, 0x07060302u);
  }
  lo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  hi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

// s_waitcnt on the vector-memory counter only (gfx9 encoding: vmcnt in bits
// 3:0 and 15:14; expcnt and lgkmcnt fields left at their maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// LDS byte address of a __shared__ pointer.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

// 128-bit LDS read issued as inline assembly.  The compiler's wait insertion
// cannot tell the LDS-DMA target of a later pipeline stage from the buffer
// being read and would drain every load in flight before an ordinary LDS
// read; these reads are instead completed by the explicit lgkmcnt waits
// below, whose register operands tie every use of a result after its wait.
template <int OFF>
__device__ __forceinline__ v4i lds_read128(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536 && OFF % 16 == 0, "ds offset");
  v4i r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "i"(OFF));
  return r;
}

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// One 16-byte-per-lane direct-to-LDS load (1 KB per wave): lane l's bytes
// land at LDS address m0 + 16 l.  The address is a 32-bit lane offset from a
// scalar base; M0 is set right before the load (nothing else in these
// kernels keeps a value in M0).  The vector-memory counter is managed by the
// explicit vmcnt waits.
struct Dma {
  uint32_t voff;
  const void* sbase;
  uint32_t m0;
};

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const Dma& d) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(d.voff), "s"(d.sbase), "s"(d.m0)
               : "memory", "m0");
}

// Token fragments of one 64-wide k stage held by one wave: MS subtiles of
// 16 tokens, two 128-bit reads per lane (k 16kg..16kg+7 and 16kg+8..16kg+15
// of token row r16).  The wave's eight packed weight tiles of the stage are
// read one by one into a rolling set of registers.
template <int MS>
struct Frag {
  v4i bx[MS][2];
};

// Wait until at most N LDS reads are outstanding; the fragment registers are
// tied so no use of them moves above the wait.
template <int N, int MS>
__device__ __forceinline__ void lgkm_wait_all(Frag<MS>& f, v4i (&q)[kWaveTiles]) {
  if constexpr (MS == 8) {
    asm volatile("s_waitcnt lgkmcnt(%24)"
                 : "+v"(f.bx[0][0]), "+v"(f.bx[0][1]), "+v"(f.bx[1][0]), "+v"(f.bx[1][1]),
                   "+v"(f.bx[2][0]), "+v"(f.bx[2][1]), "+v"(f.bx[3][0]), "+v"(f.bx[3][1]),
                   "+v"(f.bx[4][0]), "+v"(f.bx[4][1]), "+v"(f.bx[5][0]), "+v"(f.bx[5][1]),
                   "+v"(f.bx[6][0]), "+v"(f.bx[6][1]), "+v"(f.bx[7][0]), "+v"(f.bx[7][1]),
                   "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(q[4]), "+v"(q[5]),
                   "+v"(q[6]), "+v"(q[7])
                 : "i"(N));
  } else if constexpr (MS == 4) {
    asm volatile("s_waitcnt lgkmcnt(%16)"
                 : "+v"(f.bx[0][0]), "+v"(f.bx[0][1]), "+v"(f.bx[1][0]), "+v"(f.bx[1][1]),
                   "+v"(f.bx[2][0]), "+v"(f.bx[2][1]), "+v"(f.bx[3][0]), "+v"(f.bx[3][1]),
                   "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(q[4]), "+v"(q[5]),
                   "+v"(q[6]), "+v"(q[7])
                 : "i"(N));
  } else {
    static_assert(MS == 2, "token subtiles per tile: 8, 4 or 2");
    asm volatile("s_waitcnt lgkmcnt(%12)"
                 : "+v"(f.bx[0][0]), "+v"(f.bx[0][1]), "+v"(f.bx[1][0]), "+v"(f.bx[1][1]),
                   "+v"(q[0]), "+v"(q[1]), "+v"(q[2]), "+v"(q[3]), "+v"(q[4]), "+v"(q[5]),
                   "+v"(q[6]), "+v"(q[7])
                 : "i"(N));
  }
}
template <int N>
__device__ __forceinline__ void lgkm_wait_one(v4i& r) {
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(r) : "i"(N));
}

// A plain s_barrier: the waits before it are the explicit vmcnt/lgkmcnt ones
// (a full fence would drain the DMA of the stages still in flight).  The
// empty asm statements keep the compiler from moving memory accesses across.
__device__ __forceinline__ void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Per-lane LDS addresses of one ring slot: the wave's first weight tile and
// the two token chunks of row r16 (chunk c of row r is stored at chunk
// c ^ ((r >> 1) & 7)).
struct StageAddr {
  uint32_t w, x0, x1;
};

// LDS offset of the wave's j-th weight tile from its first one.  DUAL: gate
// tiles 4w..4w+3 then up tiles 16+4w..16+4w+3 (so acc[j] and acc[j+4] are
// the gate and up rows of the same H' columns); otherwise tiles 8w..8w+7.
template <bool DUAL>
__device__ __forceinline__ constexpr int wtile_off(int j) {
  return DUAL ? (j < 4 ? j : 12 + j) * 1024 : j * 1024;
}

// Chunk J of a stage: the 2*MS MFMAs of weight tile J (already widened in
// alo/ahi) with the widening of the next weight fragment qn into nlo/nhi
// interleaved (two conversion instructions behind each MFMA, so the VALU work
// co-issues with the matrix core) and this chunk's share of the ring refill.
// One asm block because the compiler clusters the conversions ahead of the
// MFMAs.  Hazards: s_nop 1 covers a VALU write of an operand right before the
// block; the last MFMAs carry no VALU, so the next block's first MFMA may read
// nlo/nhi; the accumulation chains are back-to-back MFMAs (interlocked).
constexpr uint32_t kPermHi16 = 0x07060302u;  // v_perm: upper half-words of two fp32

template <int J>
__device__ __forceinline__ void mfma_chunk(v4f (&acc)[8][8], const Frag<8>& cur, v4i alo,
                                           v4i ahi, v4i qn, v4i& nlo, v4i& nhi,
                                           const Dma (&d)[2]) {
  uint32_t o[8], t0, t1;
  asm volatile(
      "s_nop 1\n"
      "v_mfma_f32_16x16x32_bf16 %0, %34, %18, %0\n"
      "s_mov_b32 m0, %43\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %41, %42\n"
      "v_cvt_f32_i32_sdwa %16, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %1, %34, %20, %1\n"
      "v_perm_b32 %8, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %2, %34, %22, %2\n"
      "v_cvt_f32_i32_sdwa %17, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %9, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %3, %34, %24, %3\n"
      "v_cvt_f32_i32_sdwa %16, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %4, %34, %26, %4\n"
      "v_perm_b32 %10, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %5, %34, %28, %5\n"
      "v_cvt_f32_i32_sdwa %17, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %11, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %6, %34, %30, %6\n"
      "v_cvt_f32_i32_sdwa %16, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %7, %34, %32, %7\n"
      "v_perm_b32 %12, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %0, %35, %19, %0\n"
      "s_mov_b32 m0, %46\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %44, %45\n"
      "v_cvt_f32_i32_sdwa %17, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %13, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %1, %35, %21, %1\n"
      "v_cvt_f32_i32_sdwa %16, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %2, %35, %23, %2\n"
      "v_perm_b32 %14, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %3, %35, %25, %3\n"
      "v_cvt_f32_i32_sdwa %17, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %15, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %4, %35, %27, %4\n"
      "v_mfma_f32_16x16x32_bf16 %5, %35, %29, %5\n"
      "v_mfma_f32_16x16x32_bf16 %6, %35, %31, %6\n"
      "v_mfma_f32_16x16x32_bf16 %7, %35, %33, %7\n"
      : "+a"(acc[J][0]), "+a"(acc[J][1]), "+a"(acc[J][2]), "+a"(acc[J][3]), "+a"(acc[J][4]),
        "+a"(acc[J][5]), "+a"(acc[J][6]), "+a"(acc[J][7]), "=&v"(o[0]), "=&v"(o[1]),
        "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7]), "=&v"(t0),
        "=&v"(t1)
      : "v"(cur.bx[0][0]), "v"(cur.bx[0][1]), "v"(cur.bx[1][0]), "v"(cur.bx[1][1]),
        "v"(cur.bx[2][0]), "v"(cur.bx[2][1]), "v"(cur.bx[3][0]), "v"(cur.bx[3][1]),
        "v"(cur.bx[4][0]), "v"(cur.bx[4][1]), "v"(cur.bx[5][0]), "v"(cur.bx[5][1]),
        "v"(cur.bx[6][0]), "v"(cur.bx[6][1]), "v"(cur.bx[7][0]), "v"(cur.bx[7][1]), "v"(alo),
        "v"(ahi), "v"(qn[0]), "v"(qn[1]), "v"(qn[2]), "v"(qn[3]), "s"(kPermHi16),
        "v"(d[0].voff), "s"(d[0].sbase), "s"(d[0].m0), "v"(d[1].voff), "s"(d[1].sbase),
        "s"(d[1].m0)
      : "m0");
  nlo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  nhi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

template <int J>
__device__ __forceinline__ void mfma_chunk(v4f (&acc)[8][8], const Frag<8>& cur, v4i alo,
                                           v4i ahi, v4i qn, v4i& nlo, v4i& nhi,
                                           const Dma (&d)[1]) {
  uint32_t o[8], t0, t1;
  asm volatile(
      "s_nop 1\n"
      "v_mfma_f32_16x16x32_bf16 %0, %34, %18, %0\n"
      "s_mov_b32 m0, %43\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %41, %42\n"
      "v_cvt_f32_i32_sdwa %16, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %1, %34, %20, %1\n"
      "v_perm_b32 %8, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %2, %34, %22, %2\n"
      "v_cvt_f32_i32_sdwa %17, sext(%36) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %9, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %3, %34, %24, %3\n"
      "v_cvt_f32_i32_sdwa %16, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %4, %34, %26, %4\n"
      "v_perm_b32 %10, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %5, %34, %28, %5\n"
      "v_cvt_f32_i32_sdwa %17, sext(%37) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %11, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %6, %34, %30, %6\n"
      "v_cvt_f32_i32_sdwa %16, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %7, %34, %32, %7\n"
      "v_perm_b32 %12, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %0, %35, %19, %0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%38) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %13, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %1, %35, %21, %1\n"
      "v_cvt_f32_i32_sdwa %16, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %17, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %2, %35, %23, %2\n"
      "v_perm_b32 %14, %17, %16, %40\n"
      "v_cvt_f32_i32_sdwa %16, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %3, %35, %25, %3\n"
      "v_cvt_f32_i32_sdwa %17, sext(%39) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %15, %17, %16, %40\n"
      "v_mfma_f32_16x16x32_bf16 %4, %35, %27, %4\n"
      "v_mfma_f32_16x16x32_bf16 %5, %35, %29, %5\n"
      "v_mfma_f32_16x16x32_bf16 %6, %35, %31, %6\n"
      "v_mfma_f32_16x16x32_bf16 %7, %35, %33, %7\n"
      : "+a"(acc[J][0]), "+a"(acc[J][1]), "+a"(acc[J][2]), "+a"(acc[J][3]), "+a"(acc[J][4]),
        "+a"(acc[J][5]), "+a"(acc[J][6]), "+a"(acc[J][7]), "=&v"(o[0]), "=&v"(o[1]),
        "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7]), "=&v"(t0),
        "=&v"(t1)
      : "v"(cur.bx[0][0]), "v"(cur.bx[0][1]), "v"(cur.bx[1][0]), "v"(cur.bx[1][1]),
        "v"(cur.bx[2][0]), "v"(cur.bx[2][1]), "v"(cur.bx[3][0]), "v"(cur.bx[3][1]),
        "v"(cur.bx[4][0]), "v"(cur.bx[4][1]), "v"(cur.bx[5][0]), "v"(cur.bx[5][1]),
        "v"(cur.bx[6][0]), "v"(cur.bx[6][1]), "v"(cur.bx[7][0]), "v"(cur.bx[7][1]), "v"(alo),
        "v"(ahi), "v"(qn[0]), "v"(qn[1]), "v"(qn[2]), "v"(qn[3]), "s"(kPermHi16),
        "v"(d[0].voff), "s"(d[0].sbase), "s"(d[0].m0)
      : "m0");
  nlo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  nhi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

template <int J>
__device__ __forceinline__ void mfma_chunk(v4f (&acc)[8][4], const Frag<4>& cur, v4i alo,
                                           v4i ahi, v4i qn, v4i& nlo, v4i& nhi,
                                           const Dma (&d)[2]) {
  uint32_t o[8], t0, t1;
  asm volatile(
      "s_nop 1\n"
      "v_mfma_f32_16x16x32_bf16 %0, %22, %14, %0\n"
      "s_mov_b32 m0, %31\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %29, %30\n"
      "v_cvt_f32_i32_sdwa %12, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %4, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %1, %22, %16, %1\n"
      "v_cvt_f32_i32_sdwa %13, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %5, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %2, %22, %18, %2\n"
      "v_perm_b32 %6, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %13, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %7, %13, %12, %28\n"
      "v_mfma_f32_16x16x32_bf16 %3, %22, %20, %3\n"
      "v_cvt_f32_i32_sdwa %12, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %8, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %0, %23, %15, %0\n"
      "s_mov_b32 m0, %34\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %32, %33\n"
      "v_cvt_f32_i32_sdwa %13, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %9, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %1, %23, %17, %1\n"
      "v_perm_b32 %10, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %13, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %11, %13, %12, %28\n"
      "v_mfma_f32_16x16x32_bf16 %2, %23, %19, %2\n"
      "v_mfma_f32_16x16x32_bf16 %3, %23, %21, %3\n"
      : "+a"(acc[J][0]), "+a"(acc[J][1]), "+a"(acc[J][2]), "+a"(acc[J][3]), "=&v"(o[0]),
        "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]),
        "=&v"(o[7]), "=&v"(t0), "=&v"(t1)
      : "v"(cur.bx[0][0]), "v"(cur.bx[0][1]), "v"(cur.bx[1][0]), "v"(cur.bx[1][1]),
        "v"(cur.bx[2][0]), "v"(cur.bx[2][1]), "v"(cur.bx[3][0]), "v"(cur.bx[3][1]), "v"(alo),
        "v"(ahi), "v"(qn[0]), "v"(qn[1]), "v"(qn[2]), "v"(qn[3]), "s"(kPermHi16),
        "v"(d[0].voff), "s"(d[0].sbase), "s"(d[0].m0), "v"(d[1].voff), "s"(d[1].sbase),
        "s"(d[1].m0)
      : "m0");
  nlo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  nhi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

template <int J>
__device__ __forceinline__ void mfma_chunk(v4f (&acc)[8][4], const Frag<4>& cur, v4i alo,
                                           v4i ahi, v4i qn, v4i& nlo, v4i& nhi,
                                           const Dma (&d)[1]) {
  uint32_t o[8], t0, t1;
  asm volatile(
      "s_nop 1\n"
      "v_mfma_f32_16x16x32_bf16 %0, %22, %14, %0\n"
      "s_mov_b32 m0, %31\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %29, %30\n"
      "v_cvt_f32_i32_sdwa %12, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %4, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %1, %22, %16, %1\n"
      "v_cvt_f32_i32_sdwa %13, sext(%24) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %5, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %2, %22, %18, %2\n"
      "v_perm_b32 %6, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %13, sext(%25) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %7, %13, %12, %28\n"
      "v_mfma_f32_16x16x32_bf16 %3, %22, %20, %3\n"
      "v_cvt_f32_i32_sdwa %12, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %8, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_mfma_f32_16x16x32_bf16 %0, %23, %15, %0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%26) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %9, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %13, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_mfma_f32_16x16x32_bf16 %1, %23, %17, %1\n"
      "v_perm_b32 %10, %13, %12, %28\n"
      "v_cvt_f32_i32_sdwa %12, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %13, sext(%27) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %11, %13, %12, %28\n"
      "v_mfma_f32_16x16x32_bf16 %2, %23, %19, %2\n"
      "v_mfma_f32_16x16x32_bf16 %3, %23, %21, %3\n"
      : "+a"(acc[J][0]), "+a"(acc[J][1]), "+a"(acc[J][2]), "+a"(acc[J][3]), "=&v"(o[0]),
        "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]), "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]),
        "=&v"(o[7]), "=&v"(t0), "=&v"(t1)
      : "v"(cur.bx[0][0]), "v"(cur.bx[0][1]), "v"(cur.bx[1][0]), "v"(cur.bx[1][1]),
        "v"(cur.bx[2][0]), "v"(cur.bx[2][1]), "v"(cur.bx[3][0]), "v"(cur.bx[3][1]), "v"(alo),
        "v"(ahi), "v"(qn[0]), "v"(qn[1]), "v"(qn[2]), "v"(qn[3]), "s"(kPermHi16),
        "v"(d[0].voff), "s"(d[0].sbase), "s"(d[0].m0)
      : "m0");
  nlo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  nhi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

template <int J>
__device__ __forceinline__ void mfma_chunk(v4f (&acc)[8][2], const Frag<2>& cur, v4i alo,
                                           v4i ahi, v4i qn, v4i& nlo, v4i& nhi,
                                           const Dma (&d)[2]) {
  uint32_t o[8], t0, t1;
  asm volatile(
      "s_nop 1\n"
      "v_mfma_f32_16x16x32_bf16 %0, %16, %12, %0\n"
      "s_mov_b32 m0, %25\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %23, %24\n"
      "v_cvt_f32_i32_sdwa %10, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %2, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %3, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %4, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %5, %11, %10, %22\n"
      "v_mfma_f32_16x16x32_bf16 %1, %16, %14, %1\n"
      "v_cvt_f32_i32_sdwa %10, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %6, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %7, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %8, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %9, %11, %10, %22\n"
      "v_mfma_f32_16x16x32_bf16 %0, %17, %13, %0\n"
      "s_mov_b32 m0, %28\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %26, %27\n"
      "v_mfma_f32_16x16x32_bf16 %1, %17, %15, %1\n"
      : "+a"(acc[J][0]), "+a"(acc[J][1]), "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]),
        "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7]), "=&v"(t0), "=&v"(t1)
      : "v"(cur.bx[0][0]), "v"(cur.bx[0][1]), "v"(cur.bx[1][0]), "v"(cur.bx[1][1]), "v"(alo),
        "v"(ahi), "v"(qn[0]), "v"(qn[1]), "v"(qn[2]), "v"(qn[3]), "s"(kPermHi16),
        "v"(d[0].voff), "s"(d[0].sbase), "s"(d[0].m0), "v"(d[1].voff), "s"(d[1].sbase),
        "s"(d[1].m0)
      : "m0");
  nlo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  nhi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

template <int J>
__device__ __forceinline__ void mfma_chunk(v4f (&acc)[8][2], const Frag<2>& cur, v4i alo,
                                           v4i ahi, v4i qn, v4i& nlo, v4i& nhi,
                                           const Dma (&d)[1]) {
  uint32_t o[8], t0, t1;
  asm volatile(
      "s_nop 1\n"
      "v_mfma_f32_16x16x32_bf16 %0, %16, %12, %0\n"
      "s_mov_b32 m0, %25\n"
      "s_nop 0\n"
      "global_load_lds_dwordx4 %23, %24\n"
      "v_cvt_f32_i32_sdwa %10, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %2, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%18) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %3, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %4, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%19) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %5, %11, %10, %22\n"
      "v_mfma_f32_16x16x32_bf16 %1, %16, %14, %1\n"
      "v_cvt_f32_i32_sdwa %10, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %6, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%20) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %7, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_0\n"
      "v_cvt_f32_i32_sdwa %11, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_1\n"
      "v_perm_b32 %8, %11, %10, %22\n"
      "v_cvt_f32_i32_sdwa %10, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_2\n"
      "v_cvt_f32_i32_sdwa %11, sext(%21) dst_sel:DWORD dst_unused:UNUSED_PAD src0_sel:BYTE_3\n"
      "v_perm_b32 %9, %11, %10, %22\n"
      "v_mfma_f32_16x16x32_bf16 %0, %17, %13, %0\n"
      "v_mfma_f32_16x16x32_bf16 %1, %17, %15, %1\n"
      : "+a"(acc[J][0]), "+a"(acc[J][1]), "=&v"(o[0]), "=&v"(o[1]), "=&v"(o[2]), "=&v"(o[3]),
        "=&v"(o[4]), "=&v"(o[5]), "=&v"(o[6]), "=&v"(o[7]), "=&v"(t0), "=&v"(t1)
      : "v"(cur.bx[0][0]), "v"(cur.bx[0][1]), "v"(cur.bx[1][0]), "v"(cur.bx[1][1]), "v"(alo),
        "v"(ahi), "v"(qn[0]), "v"(qn[1]), "v"(qn[2]), "v"(qn[3]), "s"(kPermHi16),
        "v"(d[0].voff), "s"(d[0].sbase), "s"(d[0].m0)
      : "m0");
  nlo = v4i{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
  nhi = v4i{(int)o[4], (int)o[5], (int)o[6], (int)o[7]};
}

// After the last MFMA of a tile: wait states before the accumulators are
// read by VALU or stored (tied, so no read moves above the wait).
__device__ __forceinline__ void mfma_drain(v4f (&acc)[8][8]) {
  asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n"
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]),
                 "+a"(acc[0][4]), "+a"(acc[0][5]), "+a"(acc[0][6]), "+a"(acc[0][7]),
                 "+a"(acc[1][0]), "+a"(acc[1][1]), "+a"(acc[1][2]), "+a"(acc[1][3]),
                 "+a"(acc[1][4]), "+a"(acc[1][5]), "+a"(acc[1][6]), "+a"(acc[1][7]),
                 "+a"(acc[2][0]), "+a"(acc[2][1]), "+a"(acc[2][2]), "+a"(acc[2][3]),
                 "+a"(acc[2][4]), "+a"(acc[2][5]), "+a"(acc[2][6]), "+a"(acc[2][7]),
                 "+a"(acc[3][0]), "+a"(acc[3][1]), "+a"(acc[3][2]), "+a"(acc[3][3]),
                 "+a"(acc[3][4]), "+a"(acc[3][5]), "+a"(acc[3][6]), "+a"(acc[3][7]),
                 "+a"(acc[4][0]), "+a"(acc[4][1]), "+a"(acc[4][2]), "+a"(acc[4][3]),
                 "+a"(acc[4][4]), "+a"(acc[4][5]), "+a"(acc[4][6]), "+a"(acc[4][7]),
                 "+a"(acc[5][0]), "+a"(acc[5][1]), "+a"(acc[5][2]), "+a"(acc[5][3]),
                 "+a"(acc[5][4]), "+a"(acc[5][5]), "+a"(acc[5][6]), "+a"(acc[5][7]),
                 "+a"(acc[6][0]), "+a"(acc[6][1]), "+a"(acc[6][2]), "+a"(acc[6][3]),
                 "+a"(acc[6][4]), "+a"(acc[6][5]), "+a"(acc[6][6]), "+a"(acc[6][7]),
                 "+a"(acc[7][0]), "+a"(acc[7][1]), "+a"(acc[7][2]), "+a"(acc[7][3]),
                 "+a"(acc[7][4]), "+a"(acc[7][5]), "+a"(acc[7][6]), "+a"(acc[7][7]));
}

__device__ __forceinline__ void mfma_drain(v4f (&acc)[8][4]) {
  asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n"
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[0][2]), "+a"(acc[0][3]),
                 "+a"(acc[1][0]), "+a"(acc[1][1]), "+a"(acc[1][2]), "+a"(acc[1][3]),
                 "+a"(acc[2][0]), "+a"(acc[2][1]), "+a"(acc[2][2]), "+a"(acc[2][3]),
                 "+a"(acc[3][0]), "+a"(acc[3][1]), "+a"(acc[3][2]), "+a"(acc[3][3]),
                 "+a"(acc[4][0]), "+a"(acc[4][1]), "+a"(acc[4][2]), "+a"(acc[4][3]),
                 "+a"(acc[5][0]), "+a"(acc[5][1]), "+a"(acc[5][2]), "+a"(acc[5][3]),
                 "+a"(acc[6][0]), "+a"(acc[6][1]), "+a"(acc[6][2]), "+a"(acc[6][3]),
                 "+a"(acc[7][0]), "+a"(acc[7][1]), "+a"(acc[7][2]), "+a"(acc[7][3]));
}

__device__ __forceinline__ void mfma_drain(v4f (&acc)[8][2]) {
  asm volatile("s_nop 7\n s_nop 7\n s_nop 7\n"
               : "+a"(acc[0][0]), "+a"(acc[0][1]), "+a"(acc[1][0]), "+a"(acc[1][1]),
                 "+a"(acc[2][0]), "+a"(acc[2][1]), "+a"(acc[3][0]), "+a"(acc[3][1]),
                 "+a"(acc[4][0]), "+a"(acc[4][1]), "+a"(acc[5][0]), "+a"(acc[5][1]),
                 "+a"(acc[6][0]), "+a"(acc[6][1]), "+a"(acc[7][0]), "+a"(acc[7][1]));
}

#pragma clang diagnostic pop

// Token-fragment read I (of 2*MS) of a stage.
template <int MS, int I>
__device__ __forceinline__ void read_bx(Frag<MS>& f, const StageAddr& a) {
  if constexpr (I & 1) f.bx[I >> 1][1] = lds_read128<kWStage + (I >> 1) * 2048>(a.x1);
  else f.bx[I >> 1][0] = lds_read128<kWStage + (I >> 1) * 2048>(a.x0);
}

// One stage.  On entry: cur holds this stage's token fragments, q[1..7] this
// stage's weight tiles 1..7 and c0lo/c0hi its widened tile 0.  Chunk j runs
// the MFMAs of tile j, widens tile j+1, reads the next stage's weight tile j
// into q[j] (free since its widening in chunk j-1) and a share of its token
// fragments into nxt, and issues a share of the refill dma(j, i).  On exit
// c0lo/c0hi hold the next stage's widened tile 0.
template <bool DUAL, int MS, typename DmaFn>
__device__ __forceinline__ void stage_body(v4f (&acc)[kWaveTiles][MS], const Frag<MS>& cur,
                                           Frag<MS>& nxt, v4i (&q)[kWaveTiles],
                                           const StageAddr& a, v4i& c0lo, v4i& c0hi,
                                           DmaFn dma) {
  constexpr int NB = 2 * MS;  // token-fragment reads per stage
  v4i lo = c0lo, hi = c0hi;
  static_for<0, kWaveTiles>([&](auto jc) {
    constexpr int J = jc;
    constexpr int b0 = J * NB / kWaveTiles, b1 = (J + 1) * NB / kWaveTiles;
    if constexpr (J == kWaveTiles - 1) {
      // the next stage's tile 0, the first read of this stage, has landed
      constexpr int before = (kWaveTiles - 1) + (J * NB / kWaveTiles);
      lgkm_wait_one<(before - 1 < 15 ? before - 1 : 15)>(q[0]);
    }
    q[J] = lds_read128<wtile_off<DUAL>(J)>(a.w);
    static_for<b0, b1>([&](auto i) { read_bx<MS, i>(nxt, a); });
    v4i nlo, nhi;
    const v4i qn = J + 1 < kWaveTiles ? q[(J + 1) % kWaveTiles] : q[0];
    if constexpr (J < 4) {
      const Dma d[2] = {dma(2 * J), dma(2 * J + 1)};
      mfma_chunk<J>(acc, cur, lo, hi, qn, nlo, nhi, d);
    } else {
      const Dma d[1] = {dma(4 + J)};
      mfma_chunk<J>(acc, cur, lo, hi, qn, nlo, nhi, d);
    }
    lo = nlo;
    hi = nhi;
  });
  c0lo = lo;
  c0hi = hi;
}

// Wait until at most n whole stages of this wave's loads are in flight.
__device__ __forceinline__ void wait_stages(int n) {
  static_assert(kNStage <= 4 && kDmaPerStage * (kNStage - 1) < 64, "vmcnt immediates");
  if (n >= 2) wait_vmcnt<2 * kDmaPerStage>();
  else if (n == 1) wait_vmcnt<kDmaPerStage>();
  else wait_vmcnt<0>();
}

// The k loop of one tile over nst stages.  dma(s, i) describes load i (of
// kDmaPerStage) of stage s into ring slot s % kNStage; slot(b) gives the lane
// addresses of ring slot b.
template <bool DUAL, int MS, typename DmaFn, typename Slot>
__device__ __forceinline__ void tile_kloop(v4f (&acc)[kWaveTiles][MS], int nst, DmaFn dma,
                                           Slot slot) {
#pragma unroll
  for (int j = 0; j < kWaveTiles; ++j)
#pragma unroll
    for (int ms = 0; ms < MS; ++ms) acc[j][ms] = v4f{0.f, 0.f, 0.f, 0.f};

  const int pre = nst < kNStage ? nst : kNStage;
  for (int s = 0; s < pre; ++s)
    for (int i = 0; i < kDmaPerStage; ++i) dma16(dma(s, i));
  wait_stages(pre - 1);
  ring_barrier();  // stage 0 is in LDS for every wave

  Frag<MS> fa, fb;
  v4i q[kWaveTiles];
  v4i c0lo, c0hi;
  {
    const StageAddr a = slot(0);
    static_for<0, kWaveTiles>([&](auto j) { q[j] = lds_read128<wtile_off<DUAL>(j)>(a.w); });
    static_for<0, 2 * MS>([&](auto i) { read_bx<MS, i>(fa, a); });
  }
  lgkm_wait_all<0>(fa, q);
  i8x16_to_bf16(q[0], c0lo, c0hi);

  // iteration s: stage s+1 has landed for every wave and every wave holds
  // stage s in registers, so slot s % kNStage is refilled with stage
  // s + kNStage during the MFMAs
  int slot_next = 1 % kNStage;
  auto step = [&](int s, Frag<MS>& cur, Frag<MS>& nxt) {
    lgkm_wait_all<0>(cur, q);
    wait_stages(pre - 2);  // one refill per step: stage s+1 has pre-2 refills behind it
    ring_barrier();
    // past the end of the tile the slot is reloaded with its own stage s (a
    // harmless copy), which keeps one code path and a fixed queue depth
    const int sn = s + kNStage < nst ? s + kNStage : s;
    stage_body<DUAL, MS>(acc, cur, nxt, q, slot(slot_next), c0lo, c0hi,
                         [&](int i) { return dma(sn, i); });
    slot_next = slot_next + 1 == kNStage ? 0 : slot_next + 1;
  };
  for (int s = 0; s < nst; s += 2) {
    step(s, fa, fb);
    if (s + 1 < nst) step(s + 1, fb, fa);
  }
  // drain the trailing reads before the ring is reused
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  mfma_drain(acc);
}

// silu(g) * u with the hardware exp2 and reciprocal (relative error a few
// fp32 ulps, far below the bf16 rounding of the result)
__device__ __forceinline__ float silu_mul(float g, float u) {
  const float e = __builtin_amdgcn_exp2f(-1.4426950408889634f * g);
  return g * __builtin_amdgcn_rcpf(1.f + e) * u;
}

template <bool DUAL, int MS>
__device__ __forceinline__ void tile_epilogue(const v4f (&acc)[kWaveTiles][MS], int wave,
                                              int lane, int n0, int N, int R, int C, int p0,
                                              int nv, const int8_t* blob, uint16_t* hout,
                                              uint16_t* hout_lo, float* ybase) {
  const int r16 = lane & 15, kg = lane >> 4;
  // acc[j][ms][i] = weight row (tile base) + 4*kg + i, token p0 + ms*16 + r16
  if constexpr (DUAL) {
    const uint16_t* sig = (const uint16_t*)(blob + (size_t)3 * R * C);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int rr = n0 + (wave * 4 + j) * 16 + kg * 4;
      if (rr >= N) continue;
      float sg[4];
      {
        const uint2 sv = *(const uint2*)(sig + rr);
        sg[0] = __uint_as_float(sv.x << 16);
        sg[1] = __uint_as_float(sv.x & 0xFFFF0000u);
        sg[2] = __uint_as_float(sv.y << 16);
        sg[3] = __uint_as_float(sv.y & 0xFFFF0000u);
      }
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int tok = ms * 16 + r16;
        if (tok >= nv) continue;
        uint32_t hb[4], hl[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float gv = sg[i] * acc[j][ms][i];
          const float uv = sg[i] * acc[4 + j][ms][i];
          const float h = sg[i] * silu_mul(gv, uv);
          hb[i] = f32_to_bf16_rne(h);
          hl[i] = f32_to_bf16_rne(h - __uint_as_float(hb[i] << 16));  // the rest, for two-pass calls
        }
        uint2 pk;
        pk.x = hb[0] | (hb[1] << 16);
        pk.y = hb[2] | (hb[3] << 16);
        *(uint2*)(hout + (size_t)(p0 + tok) * R + rr) = pk;
        if (hout_lo) {
          pk.x = hl[0] | (hl[1] << 16);
          pk.y = hl[2] | (hl[3] << 16);
          *(uint2*)(hout_lo + (size_t)(p0 + tok) * R + rr) = pk;
        }
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < kWaveTiles; ++j) {
      const int cc = n0 + (wave * kWaveTiles + j) * 16 + kg * 4;
      if (cc >= N) continue;
#pragma unroll
      for (int ms = 0; ms < MS; ++ms) {
        const int tok = ms * 16 + r16;
        if (tok >= nv) continue;
        *(v4f*)(ybase + (size_t)(p0 + tok) * C + cc) = acc[j][ms];
      }
    }
  }
}

// act_lo (may be null): the low bf16 parts of the activations (act holds
// the high parts, act + act_lo the fp32 values to about 2^-16); with it every
// tile runs its k range twice, over act and then over act_lo with the same
// weights, into the same accumulators.  hout_lo (gate/up, may be null)
// receives the low bf16 parts of H' for the down GEMM's second pass.
template <bool DUAL>
__global__ __launch_bounds__(kGemmThreads) void prefill_gemm_kernel(
    int C, int R, int G, int KSmax, ExpertPool ep, int32_t* __restrict__ misc,
    const int32_t* __restrict__ offsets,
    const int32_t* __restrict__ tokpos, const uint16_t* __restrict__ act,
    const uint16_t* __restrict__ act_lo, uint16_t* __restrict__ hout,
    uint16_t* __restrict__ hout_lo, float* __restrict__ yout, size_t ysplit) {
  // LDS ring of three 48 KB slots: 32 packed tiles exactly as in HBM (1 KB
  // each), then 128 token rows x 64 bf16 with the 16-byte chunk c of row r at
  // chunk c ^ ((r >> 1) & 7): the 64 banks span two 128-byte rows, so the 16
  // rows of one read phase land on 16 distinct 16-byte bank groups.
  __shared__ __attribute__((aligned(1024))) int8_t ring[kNStage * kStageBytes];

  const int K = DUAL ? C : R;   // contraction length
  const int N = DUAL ? R : C;   // weight rows per matrix
  const int rows_per_mat = DUAL ? kTileRows / 2 : kTileRows;
  const int NT = (N + rows_per_mat - 1) / rows_per_mat;
  const int nks = K / 64;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int r16 = lane & 15, kg = lane >> 4;

  // lane addresses inside a ring slot
  const uint32_t ring_base = lds_addr(ring);
  const uint32_t wl = ring_base + (DUAL ? wave * 4 : wave * kWaveTiles) * 1024 + lane * 16;
  const uint32_t xl0 = ring_base + r16 * 128 + (((2 * kg) ^ ((r16 >> 1) & 7)) << 4);
  const uint32_t xl1 = ring_base + r16 * 128 + (((2 * kg + 1) ^ ((r16 >> 1) & 7)) << 4);
  auto slot = [&](int b) {
    const uint32_t o = (uint32_t)b * kStageBytes;
    return StageAddr{wl + o, xl0 + o, xl1 + o};
  };
  // LDS destinations of this wave's loads: packed tiles 8w..8w+7 and token
  // rows 32w..32w+31 of a slot
  const uint32_t m0_w = ring_base + wave * kWaveTiles * 1024;
  const uint32_t m0_x = ring_base + kWStage + wave * 32 * 128;

  // group tables in LDS (offsets, slots and the prefix of m-tiles of kPrefBM
  // positions over groups); the tile walk below reads them for every tile
  __shared__ int32_t s_off[MIRA_MAX_EXPERTS + 1], s_slot[MIRA_MAX_EXPERTS];
  __shared__ int32_t s_mst[MIRA_MAX_EXPERTS + 1];
  for (int i = tid; i <= G; i += kGemmThreads) {
    s_off[i] = offsets[i];
    if (i < G) s_slot[i] = ep.slot_table[i];
  }
  __syncthreads();
  if (tid < 64) {  // wave 0: each lane owns 4 consecutive groups
    int m[4], sum = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = tid * 4 + i;
      m[i] = g < G ? (s_off[g + 1] - s_off[g] + kPrefBM - 1) / kPrefBM : 0;
      sum += m[i];
    }
    int incl = sum;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(incl, off, 64);
      if (tid >= off) incl += v;
    }
    int run = incl - sum;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int g = tid * 4 + i;
      if (g < G) s_mst[g] = run;
      run += m[i];
    }
    if (tid == 63) s_mst[G] = incl;
  }
  __syncthreads();
  // k-chunks: the count (up to KSmax) whose rounds of tiles over the grid
  // take the fewest stages; ties go to fewer chunks (fewer partials)
  const int nb = gridDim.x;
  const int n_mt = s_mst[G];
  int KS = 1;
  {
    long best = -1;
    for (int ks = 1; ks <= KSmax; ++ks) {
      const long tiles = (long)n_mt * NT * ks;
      const long cost = (tiles + nb - 1) / nb * ((nks + ks - 1) / ks);
      if (best < 0 || cost < best) {
        best = cost;
        KS = ks;
      }
    }
  }
  if (!DUAL && blockIdx.x == 0 && tid == 0) misc[MISC_KSPLIT] = KS;
  const int ks_per = (nks + KS - 1) / KS;
  const int per_m = NT * KS;  // tiles per m-tile
  const int total = n_mt * per_m;

  // XCD-aware order: workgroups b, b+8, b+16, ... share an XCD, so give each
  // XCD a contiguous run of logical tiles
  const int bid = (nb % 8 == 0) ? (blockIdx.x % 8) * (nb / 8) + blockIdx.x / 8 : blockIdx.x;

  // tile tau -> (group, m-tile, k-chunk, n-tile): groups in order, m-tiles
  // fastest so the m-tiles sharing a weight tile run side by side
  struct Tile {
    int g, p0, nv, split, n0;
  };
  auto describe = [&](int tau) {
    int g = 0, hi = G;
    while (hi - g > 1) {
      const int mid = (g + hi) >> 1;
      if (s_mst[mid] * per_m <= tau) g = mid;
      else hi = mid;
    }
    const int mt_g = s_mst[g + 1] - s_mst[g];
    const int local = tau - s_mst[g] * per_m;
    const int ml = local % mt_g, rest = local / mt_g;
    const int p0 = s_off[g] + ml * kPrefBM;
    return Tile{g, p0, min(kPrefBM, s_off[g + 1] - p0), rest % KS, (rest / KS) * rows_per_mat};
  };
  // token rows of this wave's four DMA row groups: rows past the group read
  // its first row instead (their products are never stored)
  auto src_rows = [&](const Tile& t, int (&rows)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wave * 32 + i * 8 + (lane >> 3);
      const int pr = t.p0 + (r < t.nv ? r : 0);
      rows[i] = DUAL ? tokpos[pr] : pr;
    }
  };

  int rows[4] = {0, 0, 0, 0};
  if (bid < total) src_rows(describe(bid), rows);
  for (int tau = bid; tau < total; tau += nb) {
    const Tile t = describe(tau);
    const int g = t.g, p0 = t.p0, nv = t.nv, n0 = t.n0;
    const int ks0 = t.split * ks_per, ks1 = min(nks, ks0 + ks_per);
    const int nst = ks1 - ks0;
    const int slot_id = s_slot[g];
    const bool ok = slot_id >= 0 && slot_id < ep.n_slots && nst > 0;
    if (!ok && tid == 0 && ep.status && (slot_id < 0 || slot_id >= ep.n_slots))
      atomicOr(ep.status, slot_id < 0 ? 1 : 2);
    const int8_t* blob = ep.pool + (size_t)(ok ? slot_id : 0) * ep.stride;
    const int8_t* wbase = blob + (DUAL ? 0 : (size_t)2 * R * C);

    // Sources of this wave's direct-to-LDS loads: packed tiles 8w..8w+7 and
    // 4 groups of 8 token rows per stage, as 32-bit lane offsets from a
    // scalar base that advances by one stage.  Rows past the matrix read a
    // valid row instead (their products are never stored).
    uint32_t woff[kWaveTiles], xoff[4];
#pragma unroll
    for (int i = 0; i < kWaveTiles; ++i) {
      const int tl = wave * kWaveTiles + i;
      const int mat = DUAL ? (tl >> 4) : 0, rt = DUAL ? (tl & 15) : tl;
      const int row = n0 + rt * 16;
      woff[i] = (uint32_t)((size_t)mat * R * C + (size_t)((row < N ? row : n0) >> 4) * nks * 1024) +
                lane * 16;
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = wave * 32 + i * 8 + (lane >> 3);
      const int c = (lane & 7) ^ ((r >> 1) & 7);
      xoff[i] = (uint32_t)(((size_t)rows[i] * K + c * 8) * 2);
    }
    // the next tile's token rows load while this tile computes
    if (tau + nb < total) src_rows(describe(tau + nb), rows);
    if (!ok) {
      // A missing expert contributes nothing: its partial outputs are zero,
      // so the combine (which sums every position's partials) leaves its term
      // out.  Its H' rows stay unwritten; only this GEMM would read them.
      if (!DUAL) {
        float* yb = yout + (size_t)t.split * ysplit;
        const int q4 = min(kTileRows, N - n0) / 4;
        for (int i = tid; i < nv * q4; i += kGemmThreads)
          *(v4f*)(yb + (size_t)(p0 + i / q4) * C + n0 + (i % q4) * 4) = v4f{0.f, 0.f, 0.f, 0.f};
      }
      continue;
    }

    const int8_t* wstage0 = wbase + (size_t)ks0 * 1024;
    const int8_t* xstage0 = (const int8_t*)(act + (size_t)ks0 * 64);
    const int8_t* xstage0_lo = act_lo ? (const int8_t*)(act_lo + (size_t)ks0 * 64) : xstage0;
    // load i of stage s: packed tiles for i < 8, token row groups after;
    // stages nst .. 2*nst-1 (two-pass calls) repeat the weights over act_lo
    auto dma = [&](int s, int i) {
      const uint32_t so = (uint32_t)(s % kNStage) * kStageBytes;
      const bool lo = s >= nst;
      const int sk = lo ? s - nst : s;
      if (i < kWaveTiles) return Dma{woff[i], wstage0 + (size_t)sk * 1024, m0_w + so + i * 1024};
      const int r = i - kWaveTiles;
      return Dma{xoff[r], (lo ? xstage0_lo : xstage0) + (size_t)sk * 128, m0_x + so + r * 1024};
    };
    const int nst_all = act_lo ? 2 * nst : nst;

    // every wave is done with the ring before it is refilled.  The previous
    // tile's stores may still be in flight: the counter waits below count
    // only this tile's loads, and as the counter retires in issue order the
    // older stores only make them stricter.
    ring_barrier();

    float* ybase = DUAL ? nullptr : yout + (size_t)t.split * ysplit;
    // token subtiles actually present: the group's last tile runs a shorter
    // loop when it holds at most 64 or 32 tokens
    if (nv > 64) {
      v4f acc[kWaveTiles][8];
      tile_kloop<DUAL, 8>(acc, nst_all, dma, slot);
      tile_epilogue<DUAL, 8>(acc, wave, lane, n0, N, R, C, p0, nv, blob, hout, hout_lo, ybase);
    } else if (nv > 32) {
      v4f acc[kWaveTiles][4];
      tile_kloop<DUAL, 4>(acc, nst_all, dma, slot);
      tile_epilogue<DUAL, 4>(acc, wave, lane, n0, N, R, C, p0, nv, blob, hout, hout_lo, ybase);
    } else {
      v4f acc[kWaveTiles][2];
      tile_kloop<DUAL, 2>(acc, nst_all, dma, slot);
      tile_epilogue<DUAL, 2>(acc, wave, lane, n0, N, R, C, p0, nv, blob, hout, hout_lo, ybase);
    }
  }
}

// out[t][c] = sum_j w[t][j] * Y[inv[t*k+j]][c] + sum_s Y[inv[T*k + s*T + t]][c],
// each Y the ordered sum of its KS k-chunk partials (KS chosen by the down
// GEMM and read from misc)
__global__ __launch_bounds__(256) void combine_kernel(int T, int C, int k, int S,
                                                      const int32_t* __restrict__ misc,
                                                      size_t ysplit,
                                                      const int32_t* __restrict__ inv,
                                                      const float* __restrict__ wts,
                                                      const float* __restrict__ y,
                                                      float* __restrict__ out) {
  const int t = blockIdx.y;
  const int c = (blockIdx.x * 256 + threadIdx.x) * 4;
  if (c >= C) return;
  const int KS = misc[MISC_KSPLIT];
  auto yrow = [&](size_t pos) {
    v4f v = *(const v4f*)(y + pos * C + c);
    for (int sp = 1; sp < KS; ++sp) v += *(const v4f*)(y + sp * ysplit + pos * C + c);
    return v;
  };
  v4f s = {0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < k; ++j) s += wts[(size_t)t * k + j] * yrow(inv[(size_t)t * k + j]);
  for (int sh = 0; sh < S; ++sh) s += yrow(inv[(size_t)T * k + (size_t)sh * T + t]);
  *(v4f*)(out + (size_t)t * C + c) = s;
}

// fp32 activations as two bf16 parts: hi = bf16(x), lo = bf16(x - hi)
__global__ __launch_bounds__(256) void f32_to_bf16_pair_kernel(const float* __restrict__ x,
                                                               uint16_t* __restrict__ hi,
                                                               uint16_t* __restrict__ lo, size_t n) {
  for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256) {
    const uint32_t h = f32_to_bf16_rne(x[i]);
    hi[i] = (uint16_t)h;
    lo[i] = (uint16_t)f32_to_bf16_rne(x[i] - __uint_as_float(h << 16));
  }
}

// Workgroups of kernel k that fit on one CU, queried once per process (the
// first caller fills the cache; concurrent callers wait for it).
template <typename Kern>
static int gemm_occupancy(Kern k, std::once_flag& once, int& occ) {
  std::call_once(once, [&] {
    int o = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&o, k, kGemmThreads, 0) != hipSuccess || o < 1)
      o = 1;
    occ = o;
  });
  return occ;
}

static int persistent_grid(int occ, long max_tiles) {
  long cap = (long)device_cu_count() * occ;
  if (max_tiles < cap) cap = max_tiles < 8 ? max_tiles : max_tiles / 8 * 8;
  return (int)(cap < 1 ? 1 : cap);
}

hipError_t launch_prefill(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                          const ExpertPool& ep, float* out, hipStream_t st) {
  const int T = L.T;
  if (T == 0) return hipSuccess;
  // fp32 activations run both GEMMs in two passes (high and low bf16 parts
  // of x, then of H'), bf16 activations in one
  const uint16_t* xb = (const uint16_t*)x;
  const uint16_t* xlo = nullptr;
  uint16_t* hlo = nullptr;
  if (s.act_dtype == MIRA_F32) {
    const size_t n = (size_t)T * L.C;
    const int blocks = (int)((n + 255) / 256 < 4096 ? (n + 255) / 256 : 4096);
    launch_timed("prefill_cvt", f32_to_bf16_pair_kernel, dim3(blocks), dim3(256), 0, st,
                 (const float*)x, w.xb16, w.xlo16, n);
    xb = w.xb16;
    xlo = w.xlo16;
    hlo = w.hlo;
  }
  const size_t ysplit = (size_t)L.P * L.C;
  {
    auto kern = prefill_gemm_kernel<true>;
    static std::once_flag once;
    static int occ = 0;
    const long tiles = (long)L.mt_max * ((L.R + kTileRows / 2 - 1) / (kTileRows / 2));
    const int grid = persistent_grid(gemm_occupancy(kern, once, occ), tiles);
    launch_timed("prefill_gateup", kern, dim3(grid), dim3(kGemmThreads), 0, st, L.C, L.R, L.G, 1,
                 ep, w.misc, w.offsets, w.tokpos, xb, xlo, w.hbuf, hlo, (float*)nullptr, (size_t)0);
  }
  {
    auto kern = prefill_gemm_kernel<false>;
    static std::once_flag once;
    static int occ = 0;
    const long tiles = (long)L.mt_max * ((L.C + kTileRows - 1) / kTileRows) * L.ksplit;
    const int grid = persistent_grid(gemm_occupancy(kern, once, occ), tiles);
    launch_timed("prefill_down", kern, dim3(grid), dim3(kGemmThreads), 0, st, L.C, L.R, L.G,
                 L.ksplit, ep, w.misc, w.offsets, w.tokpos, (const uint16_t*)w.hbuf,
                 (const uint16_t*)hlo, (uint16_t*)nullptr, (uint16_t*)nullptr, w.ybuf, ysplit);
  }
  {
    dim3 grid((L.C / 4 + 255) / 256, T);
    launch_timed("prefill_combine", combine_kernel, grid, dim3(256), 0, st, T, L.C, L.k, L.S,
                 (const int32_t*)w.misc, ysplit, w.inv, w.wts, w.ybuf, out);
  }
  return hipGetLastError();
}

}  // namespace mira
