// Internal declarations shared by the HIP kernels and the host entry points.
#pragma once

#include <hip/hip_runtime.h>
#include <hip/hip_ext.h>
#include <stddef.h>
#include <stdint.h>

#include "mira.h"

namespace mira {

// ---------------------------------------------------------------------------
// Compile-time tiling constants
// ---------------------------------------------------------------------------
constexpr int kDigits = 3;           // base-256 digits of a fixed-point activation x
constexpr int kFixBits = 22;         // |fixed-point x| < 2^22
constexpr int kBlk = 64;             // rows of H' sharing one fixed-point exponent
constexpr int kTokPerGroup = 5;      // tokens per 16-column MFMA operand of x (3 digits each)
constexpr int kDecodeMaxGroups = (MIRA_DECODE_MAX_TOKENS + kTokPerGroup - 1) / kTokPerGroup;
// H' (the down projection's input) is written as three digits (kFixBits) when
// one x group covers the call (T <= kTokPerGroup) and as two digits of
// kHFixBits2 bits otherwise, so that an operand of H' holds 8 tokens instead
// of 5 and the down kernel needs half the token groups.
constexpr int kHFixBits2 = 14;       // two digits: |fixed-point H'| <= 2^14 (digits stay in int8)
__host__ __device__ constexpr int h_digits(int x_groups) { return x_groups == 1 ? 3 : 2; }
__host__ __device__ constexpr int h_tok_per_group(int hd) { return hd == 3 ? 5 : 8; }
constexpr int kPrefBM = 128;         // prefill tile: tokens per m-tile (shared by both GEMMs)

inline __host__ __device__ size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// Packed int8 matrices [rows][K] are stored as 16-row x 64-column tiles of
// 1024 bytes, row-of-tiles major; inside a tile, 16-byte run g*16 + i holds
// row i, columns 16g .. 16g+15.  One wave's 128-bit loads of a tile are one
// contiguous kilobyte and land exactly in the int8 MFMA operand layout
// (lane l = row l%16, k-group l/16).
inline __host__ __device__ size_t tiled_offset(size_t r, size_t k, size_t K) {
  return (((r >> 4) * (K >> 6) + (k >> 6)) << 10) + ((((k & 63) >> 4) << 4 | (r & 15)) << 4) +
         (k & 15);
}

// ---------------------------------------------------------------------------
// Workspace layout of one call with T tokens.  Every region is 256-aligned.
// Decode regions are sized for min(T, MIRA_DECODE_MAX_TOKENS) tokens.
// ---------------------------------------------------------------------------
struct Layout {
  int T, E, S, G, k, C, R;
  int P;        // (token, slot) pairs: T*k + S*T
  int Pd;       // pairs of the decode sizing
  int Td;       // tokens of the decode sizing
  int mt_max;   // upper bound of prefill m-tiles
  int ksplit;   // most k-chunks of the prefill down GEMM (partials summed in order by the combine)
  size_t logits, idx, wts, counts, offsets, inv, tokpos, wpos, misc, active, mstart, pcnt,
      dwork, xdig, hdig, hexp, xb16, xlo16, hbuf, hlo, ybuf, total;
};

// One non-empty expert group of a decode call, written by the decode
// preparation kernel so that each expert kernel starts from a single load.
struct DecodeWork {
  int32_t group;  // expert (routed 0..E-1, shared E..E+S-1); -1 = no work
  int32_t slot;   // slot seen by the routing; the gate/up kernel replaces it with the slot it
                  // resolved from the table (-1 if invalid), which the down kernel uses
  int32_t off;    // first permuted position of the group
  int32_t n;      // positions (tokens) of the group, <= MIRA_DECODE_MAX_TOKENS
  int32_t tok[MIRA_DECODE_MAX_TOKENS];  // token of position off+i
  int32_t xe[MIRA_DECODE_MAX_TOKENS];   // fixed-point exponent of that token's x
  float w[MIRA_DECODE_MAX_TOKENS];      // combine weight of position off+i
};

// Largest number of (token, slot) pairs the decode preparation handles.
constexpr int kDecodeMaxPairs = 1024;

// The prefill permutation runs in chunks of kPermChunk routed pairs, one
// workgroup each, when there are 2..kPermChunkMax chunks (one workgroup
// otherwise).
constexpr int kPermChunk = 1024;
constexpr int kPermChunkMax = 64;

// misc[] slots (int32)
enum : int { MISC_NACTIVE = 0, MISC_MTOTAL = 1, MISC_KSPLIT = 2, MISC_COUNT = 16 };

// Most k-chunks the prefill down GEMM may split its contraction (R) into
// (the workspace holds that many fp32 partial outputs); the kernel picks the
// count that best fills the grid for the actual routing.
inline int prefill_ksplit(int R) {
  const int s = R / 4096;
  return s < 1 ? 1 : (s > 4 ? 4 : s);
}

inline int decode_max_active_of(int G, int T, int k, int S) {
  const int pairs_groups = T * k + S;
  return G < pairs_groups ? G : pairs_groups;
}

inline Layout make_layout(const mira_shape& s, int T) {
  Layout L{};
  L.T = T;
  L.E = s.n_experts;
  L.S = s.n_shared;
  L.G = s.n_experts + s.n_shared;
  L.k = s.top_k;
  L.C = s.hidden;
  L.R = s.ffn;
  L.P = T * s.top_k + s.n_shared * T;
  L.Td = T < MIRA_DECODE_MAX_TOKENS ? T : MIRA_DECODE_MAX_TOKENS;
  L.Pd = L.Td * s.top_k + s.n_shared * L.Td;
  L.mt_max = L.P / kPrefBM + L.G + 1;
  L.ksplit = prefill_ksplit(s.ffn);
  size_t o = 0;
  auto take = [&](size_t bytes) {
    size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  const size_t P = (size_t)L.P, G = (size_t)L.G, Tz = (size_t)T;
  L.logits = take(Tz * L.E * 4);
  L.idx = take(Tz * L.k * 4);
  L.wts = take(Tz * L.k * 4);
  L.counts = take(G * 4);
  L.offsets = take((G + 1) * 4);
  L.inv = take(P * 4);
  L.tokpos = take(P * 4);
  L.wpos = take(P * 4);
  L.misc = take(MISC_COUNT * 4);
  L.active = take(G * 4);
  L.mstart = take((G + 1) * 4);
  L.pcnt = take((size_t)kPermChunkMax * L.E * 4);
  L.dwork = take(G * sizeof(DecodeWork));
  L.xdig = take((size_t)L.Td * kDigits * L.C);
  L.hdig = take((size_t)L.Pd * kDigits * L.R);  // room for three digits
  // H' exponents: one per 64-row block, or per 16-row tile for one token
  L.hexp = take((size_t)L.Pd * (L.Td == 1 ? L.R / 16 : L.R / kBlk) * 4);
  // fp32 activations: x and H' as high and low bf16 parts (two-pass GEMMs)
  const bool f32 = s.act_dtype == MIRA_F32;
  L.xb16 = take(f32 ? Tz * L.C * 2 : 0);
  L.xlo16 = take(f32 ? Tz * L.C * 2 : 0);
  L.hbuf = take(P * L.R * 2);
  L.hlo = take(f32 ? P * L.R * 2 : 0);
  L.ybuf = take((size_t)L.ksplit * P * L.C * 4);
  L.total = o;
  return L;
}

// Device pointers of one call's workspace regions.
struct WsPtr {
  float* logits;
  int32_t* idx;
  float* wts;
  int32_t* counts;
  int32_t* offsets;
  int32_t* inv;
  int32_t* tokpos;
  float* wpos;
  int32_t* misc;
  int32_t* active;
  int32_t* mstart;
  int32_t* pcnt;
  DecodeWork* dwork;
  int8_t* xdig;
  int8_t* hdig;
  int32_t* hexp;
  uint16_t* xb16;
  uint16_t* xlo16;
  uint16_t* hbuf;
  uint16_t* hlo;
  float* ybuf;
};

inline WsPtr ws_ptrs(const Layout& L, void* base) {
  char* b = (char*)base;
  WsPtr w;
  w.logits = (float*)(b + L.logits);
  w.idx = (int32_t*)(b + L.idx);
  w.wts = (float*)(b + L.wts);
  w.counts = (int32_t*)(b + L.counts);
  w.offsets = (int32_t*)(b + L.offsets);
  w.inv = (int32_t*)(b + L.inv);
  w.tokpos = (int32_t*)(b + L.tokpos);
  w.wpos = (float*)(b + L.wpos);
  w.misc = (int32_t*)(b + L.misc);
  w.active = (int32_t*)(b + L.active);
  w.mstart = (int32_t*)(b + L.mstart);
  w.pcnt = (int32_t*)(b + L.pcnt);
  w.dwork = (DecodeWork*)(b + L.dwork);
  w.xdig = (int8_t*)(b + L.xdig);
  w.hdig = (int8_t*)(b + L.hdig);
  w.hexp = (int32_t*)(b + L.hexp);
  w.xb16 = (uint16_t*)(b + L.xb16);
  w.xlo16 = (uint16_t*)(b + L.xlo16);
  w.hbuf = (uint16_t*)(b + L.hbuf);
  w.hlo = (uint16_t*)(b + L.hlo);
  w.ybuf = (float*)(b + L.ybuf);
  return w;
}

inline int decode_max_active(const Layout& L) { return decode_max_active_of(L.G, L.T, L.k, L.S); }

// Everything the expert kernels need to find a packed expert.
struct ExpertPool {
  const int8_t* pool;
  const int32_t* slot_table;
  uint64_t stride;
  int32_t n_slots;
  int32_t* status;  // may be null
};

// ---------------------------------------------------------------------------
// Host-side launch helpers (defined in the .hip files)
// ---------------------------------------------------------------------------
// Kernel timing hooks (mira_api.cpp); no-ops unless profiling is enabled.
void prof_begin(const char* name, hipStream_t st);
void prof_end(const char* name, hipStream_t st);
// Events for one timed launch of kernel `name` (both null unless profiling
// selects it); the dispatch packet itself records them, so the interval is
// the kernel's own start and end.
void prof_events(const char* name, hipEvent_t* start, hipEvent_t* stop);

template <typename... Args, typename F = void (*)(Args...)>
inline void launch_timed(const char* name, F kernel, dim3 grid, dim3 block, uint32_t shmem,
                         hipStream_t st, Args... args) {
  hipEvent_t a = nullptr, b = nullptr;
  prof_events(name, &a, &b);
  hipExtLaunchKernelGGL(kernel, grid, block, shmem, st, a, b, 0, args...);
}

hipError_t launch_route(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                        const void* wr, const float* bias, float* logits_out, hipStream_t st);
hipError_t launch_permute(const Layout& L, const WsPtr& w,
                          const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                          float* wts_out, int32_t* offsets_out, int32_t* order_out,
                          hipStream_t st);
hipError_t launch_decode_prep(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                              const void* wr, const float* bias, float* logits_out,
                              const ExpertPool& ep, int32_t* counts_out, int32_t* idx_out,
                              float* wts_out, int32_t* offsets_out, int32_t* order_out,
                              hipStream_t st);
hipError_t launch_decode(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                         const ExpertPool& ep, float* out, hipStream_t st);
hipError_t launch_prefill(const mira_shape& s, const Layout& L, const WsPtr& w, const void* x,
                          const ExpertPool& ep, float* out, hipStream_t st);
hipError_t launch_pack_i4(int C, int R, int n, int w_dtype, const void* wg, const void* wu,
                          const void* wd, float eps, void* packed, uint64_t stride, hipStream_t st);
hipError_t launch_pack(int C, int R, int n, int w_dtype, const void* wg, const void* wu,
                       const void* wd, float eps, void* packed, uint64_t stride, hipStream_t st);
hipError_t launch_predict(const mira_pred_shape& p, const void* x, int T, const void* w1,
                          const float* b1, const void* w2, const float* b2, float* scores,
                          void* ws, hipStream_t st);
size_t mixture_ws_bytes(int n_groups, const mira_mixture_shape& p);
hipError_t launch_mixture(const mira_mixture_shape& p, const mira_mixture_weights& w,
                          const void* x, const float* logits, const int32_t* topk_idx, int T,
                          float* probs, float* alpha, void* ws, hipStream_t st);
hipError_t launch_set_slot(int32_t* table, int expert, int slot, hipStream_t st);
// Device address of the library's scratch array on the current device
// (noalloc.hip), looked up on the first call per device.
hipError_t noalloc_scratch(void** ptr);

int device_cu_count();

// The thread-local message behind mira_last_error (mira_api.cpp): set_error
// stores a formatted message and returns code; clear_error empties it and
// returns MIRA_OK.
int set_error(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int clear_error();

}  // namespace mira
