// Host entry points of the C ABI declared in include/mira.h: argument
// checks, workspace layout, path dispatch, the host packer, expert staging
// and kernel timing.  Every check runs before any launch.
#include <hip/hip_runtime.h>
#include <sched.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "mira.h"
#include "int4_format.h"
#include "mira_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return MIRA_OK;
}

#define HIP_TRY(call)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (call);                                                            \
    if (e_ != hipSuccess)                                                              \
      return fail(MIRA_ERR_HIP, "%s failed: %s", #call, hipGetErrorString(e_));       \
  } while (0)

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

int check_shape(const mira_shape* s) {
  if (!s) return fail(MIRA_ERR_ARG, "shape is NULL");
  if (s->reserved != 0) return fail(MIRA_ERR_ARG, "shape.reserved must be 0");
  if (s->hidden <= 0 || s->hidden % 64)
    return fail(MIRA_ERR_SHAPE, "hidden (%d) must be a positive multiple of 64", s->hidden);
  if (s->ffn <= 0 || s->ffn % 64)
    return fail(MIRA_ERR_SHAPE, "ffn (%d) must be a positive multiple of 64", s->ffn);
  if (s->n_experts < 1) return fail(MIRA_ERR_SHAPE, "n_experts must be >= 1");
  if (s->n_shared < 0) return fail(MIRA_ERR_SHAPE, "n_shared must be >= 0");
  if (s->n_experts + s->n_shared > MIRA_MAX_EXPERTS)
    return fail(MIRA_ERR_SHAPE, "n_experts + n_shared must be <= %d", MIRA_MAX_EXPERTS);
  if (s->top_k < 1 || s->top_k > s->n_experts || s->top_k > MIRA_MAX_TOPK)
    return fail(MIRA_ERR_SHAPE, "top_k (%d) must be in [1, min(n_experts, %d)]", s->top_k,
                MIRA_MAX_TOPK);
  if (s->act_dtype != MIRA_F32 && s->act_dtype != MIRA_BF16)
    return fail(MIRA_ERR_ARG, "act_dtype must be MIRA_F32 or MIRA_BF16");
  const uint32_t known =
      MIRA_FLAG_SOFTMAX_ALL | MIRA_FLAG_FORCE_DECODE | MIRA_FLAG_FORCE_PREFILL | MIRA_FLAG_INT4;
  if (s->flags & ~known) return fail(MIRA_ERR_ARG, "unknown flag bits 0x%x", s->flags & ~known);
  if ((s->flags & MIRA_FLAG_FORCE_DECODE) && (s->flags & MIRA_FLAG_FORCE_PREFILL))
    return fail(MIRA_ERR_ARG, "FORCE_DECODE and FORCE_PREFILL are exclusive");
  // largest byte offsets must fit comfortably
  const double rc = (double)s->hidden * (double)s->ffn;
  if (rc * 3 > 4.0e18) return fail(MIRA_ERR_SHAPE, "expert too large");
  return MIRA_OK;
}

bool decode_fits(const mira_shape& s, int T) {
  return T <= MIRA_DECODE_MAX_TOKENS && T * (s.top_k + s.n_shared) <= mira::kDecodeMaxPairs;
}

bool use_decode(const mira_shape& s, int T) {
  if (s.flags & (MIRA_FLAG_FORCE_DECODE | MIRA_FLAG_INT4)) return true;
  if (s.flags & MIRA_FLAG_FORCE_PREFILL) return false;
  return decode_fits(s, T);
}

int check_args(const mira_shape* s, const mira_moe_args* a, mira::Layout* L) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (!a) return fail(MIRA_ERR_ARG, "args is NULL");
  if (a->n_tokens < 0) return fail(MIRA_ERR_SHAPE, "n_tokens must be >= 0");
  if ((s->flags & MIRA_FLAG_FORCE_DECODE) && !decode_fits(*s, a->n_tokens))
    return fail(MIRA_ERR_SHAPE,
                "FORCE_DECODE needs n_tokens <= %d and n_tokens * (top_k + n_shared) <= %d "
                "(got %d tokens)", MIRA_DECODE_MAX_TOKENS, mira::kDecodeMaxPairs, a->n_tokens);
  if ((int64_t)a->n_tokens * (s->top_k + s->n_shared) > (int64_t)1 << 30)
    return fail(MIRA_ERR_SHAPE, "too many tokens");
  const bool i4 = s->flags & MIRA_FLAG_INT4;
  if (i4 && (s->hidden % 128 || s->ffn % 128))
    return fail(MIRA_ERR_SHAPE, "INT4 experts need hidden and ffn multiples of 128");
  if (i4 && (s->flags & MIRA_FLAG_FORCE_PREFILL))
    return fail(MIRA_ERR_UNSUPPORTED, "INT4 experts run on the decode kernels only");
  if (i4 && !decode_fits(*s, a->n_tokens))
    return fail(MIRA_ERR_UNSUPPORTED,
                "INT4 experts run on the decode kernels only: n_tokens <= %d and n_tokens * "
                "(top_k + n_shared) <= %d (got %d tokens)", MIRA_DECODE_MAX_TOKENS,
                mira::kDecodeMaxPairs, a->n_tokens);
  const size_t expert_bytes = i4 ? mira_packed_expert_bytes_int4(s->hidden, s->ffn)
                                 : mira_packed_expert_bytes(s->hidden, s->ffn);
  *L = mira::make_layout(*s, a->n_tokens);
  if (a->n_tokens == 0) return MIRA_OK;
  if (!a->x || !a->w_router || !a->slot_table || !a->slot_pool || !a->out || !a->workspace)
    return fail(MIRA_ERR_ARG, "x, w_router, slot_table, slot_pool, out and workspace are required");
  if (a->n_slots < 1) return fail(MIRA_ERR_ARG, "n_slots must be >= 1");
  if (!aligned(a->x, 16) || !aligned(a->w_router, 16) || !aligned(a->out, 16))
    return fail(MIRA_ERR_ALIGN, "x, w_router and out must be 16-byte aligned");
  if (!aligned(a->slot_pool, 256) || a->slot_stride % 256)
    return fail(MIRA_ERR_ALIGN, "slot_pool and slot_stride must be 256-byte aligned");
  if (a->slot_stride < expert_bytes)
    return fail(MIRA_ERR_SHAPE, "slot_stride %llu smaller than a packed expert (%zu bytes)",
                (unsigned long long)a->slot_stride, expert_bytes);
  if (!aligned(a->workspace, 256)) return fail(MIRA_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (a->workspace_bytes < L->total)
    return fail(MIRA_ERR_WORKSPACE, "workspace has %llu bytes, %zu needed for %d tokens",
                (unsigned long long)a->workspace_bytes, L->total, a->n_tokens);
  return MIRA_OK;
}

mira::ExpertPool pool_of(const mira_moe_args* a) {
  mira::ExpertPool ep;
  ep.pool = (const int8_t*)a->slot_pool;
  ep.slot_table = a->slot_table;
  ep.stride = a->slot_stride;
  ep.n_slots = a->n_slots;
  ep.status = a->status;
  return ep;
}

int run_route(const mira_shape* s, const mira_moe_args* a, const mira::Layout& L, hipStream_t st) {
  mira::WsPtr w = mira::ws_ptrs(L, a->workspace);
  if (use_decode(*s, L.T)) {
    // one workgroup: router, top-k, permutation and the digits of x
    HIP_TRY(mira::launch_decode_prep(*s, L, w, a->x, a->w_router, a->router_bias, a->logits,
                                     pool_of(a), a->expert_counts, a->topk_idx, a->topk_weight,
                                     a->expert_offsets, a->pair_order, st));
    return MIRA_OK;
  }
  HIP_TRY(mira::launch_route(*s, L, w, a->x, a->w_router, a->router_bias, a->logits, st));
  HIP_TRY(mira::launch_permute(L, w, pool_of(a), a->expert_counts, a->topk_idx,
                               a->topk_weight, a->expert_offsets, a->pair_order, st));
  return MIRA_OK;
}

int run_experts(const mira_shape* s, const mira_moe_args* a, const mira::Layout& L,
                hipStream_t st) {
  mira::WsPtr w = mira::ws_ptrs(L, a->workspace);
  if (use_decode(*s, L.T))
    HIP_TRY(mira::launch_decode(*s, L, w, a->x, pool_of(a), a->out, st));
  else
    HIP_TRY(mira::launch_prefill(*s, L, w, a->x, pool_of(a), a->out, st));
  return MIRA_OK;
}

// ---- host packer ---------------------------------------------------------
int host_threads() {
  cpu_set_t set;
  if (sched_getaffinity(0, sizeof(set), &set) == 0) {
    const int n = CPU_COUNT(&set);
    if (n > 0) return n;
  }
  const unsigned h = std::thread::hardware_concurrency();
  return h ? (int)h : 1;
}

template <typename F>
void parallel_for(int64_t n, F&& f) {
  const int nt = (int)std::min<int64_t>(host_threads(), std::max<int64_t>(1, n));
  if (nt <= 1) {
    f(0, n);
    return;
  }
  std::vector<std::thread> th;
  const int64_t chunk = (n + nt - 1) / nt;
  for (int i = 0; i < nt; ++i) {
    const int64_t b = i * chunk, e = std::min(n, b + chunk);
    if (b >= e) break;
    th.emplace_back([&f, b, e] { f(b, e); });
  }
  for (auto& t : th) t.join();
}

inline float h_bf16_to_f32(uint16_t b) {
  uint32_t u = (uint32_t)b << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

inline uint16_t h_f32_to_bf16_rne(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename WT>
inline float h_ld(const WT* p, size_t i);
template <>
inline float h_ld<float>(const float* p, size_t i) { return p[i]; }
template <>
inline float h_ld<uint16_t>(const uint16_t* p, size_t i) { return h_bf16_to_f32(p[i]); }

inline int8_t h_quant(float w, float sigma) {
  float q = std::rint(w / sigma);
  q = std::fmin(std::fmax(q, -127.f), 127.f);
  return (int8_t)(int)q;
}

template <typename WT>
void host_pack_one(int C, int R, const WT* wg, const WT* wu, const WT* wd, float eps,
                   int8_t* blob, uint64_t stride) {
  std::vector<float> alpha(R, 0.f);
  parallel_for(R, [&](int64_t b, int64_t e) {
    for (int64_t r = b; r < e; ++r) {
      float m = 0.f;
      for (int c = 0; c < C; ++c) {
        m = std::fmax(m, std::fabs(h_ld(wg, (size_t)r * C + c)));
        m = std::fmax(m, std::fabs(h_ld(wu, (size_t)r * C + c)));
      }
      alpha[r] = m;
    }
  });
  parallel_for(R, [&](int64_t b, int64_t e) {
    for (int c = 0; c < C; ++c)
      for (int64_t r = b; r < e; ++r)
        alpha[r] = std::fmax(alpha[r], std::fabs(h_ld(wd, (size_t)c * R + r)));
  });
  std::vector<uint16_t> sbits(R);
  std::vector<float> sigma(R);
  for (int r = 0; r < R; ++r) {
    const float s32 = std::fmax(alpha[r], eps) / 127.0f;
    sbits[r] = h_f32_to_bf16_rne(s32);
    sigma[r] = h_bf16_to_f32(sbits[r]);
  }
  parallel_for((int64_t)2 * R, [&](int64_t b, int64_t e) {
    for (int64_t i = b; i < e; ++i) {
      const int mat = (int)(i / R), r = (int)(i % R);
      const WT* src = (mat == 0 ? wg : wu) + (size_t)r * C;
      int8_t* dst = blob + (size_t)mat * R * C;
      for (int c = 0; c < C; ++c) dst[mira::tiled_offset(r, c, C)] = h_quant(h_ld(src, c), sigma[r]);
    }
  });
  parallel_for(C, [&](int64_t b, int64_t e) {
    int8_t* dst = blob + (size_t)2 * R * C;
    for (int64_t c = b; c < e; ++c)
      for (int r = 0; r < R; ++r)
        dst[mira::tiled_offset(c, r, R)] = h_quant(h_ld(wd, (size_t)c * R + r), sigma[r]);
  });
  uint8_t* sig = (uint8_t*)(blob + (size_t)3 * R * C);
  for (int r = 0; r < R; ++r) {
    sig[2 * r] = (uint8_t)(sbits[r] & 0xFF);
    sig[2 * r + 1] = (uint8_t)(sbits[r] >> 8);
  }
  const uint64_t used = (uint64_t)3 * R * C + (uint64_t)2 * R;
  if (stride > used) std::memset(blob + used, 0, stride - used);
}

// ---- kernel timing ---------------------------------------------------------
struct ProfRec {
  const char* name;
  hipEvent_t a, b;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::string g_prof_only;
std::vector<ProfRec> g_prof;
std::vector<hipEvent_t> g_prof_free;

hipEvent_t prof_event() {
  if (!g_prof_free.empty()) {
    hipEvent_t e = g_prof_free.back();
    g_prof_free.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// INT4 variant, one (matrix, row) per work item; the same arithmetic as the
// device packer (fp32 division, round half to even, fp16 scale rules).
template <typename WT>
void host_pack_one_i4(int C, int R, const WT* wg, const WT* wu, const WT* wd, float eps,
                      uint8_t* blob, uint64_t stride) {
  parallel_for((int64_t)2 * R + C, [&](int64_t b, int64_t e) {
    for (int64_t it = b; it < e; ++it) {
      const int mat = it < R ? 0 : it < 2 * R ? 1 : 2;
      const int r = (int)(mat == 0 ? it : mat == 1 ? it - R : it - 2 * R);
      const int K = mat == 2 ? R : C;
      const WT* src = (mat == 0 ? wg : mat == 1 ? wu : wd) + (size_t)r * K;
      uint8_t* m = blob + (size_t)mat * mira::i4_matrix_bytes(R, C);
      for (int blk = 0; blk < K / 64; ++blk) {
        float w[64], alpha = 0.f;
        for (int c = 0; c < 64; ++c) {
          w[c] = h_ld(src, (size_t)blk * 64 + c);
          alpha = std::fmax(alpha, std::fabs(w[c]));
        }
        const uint16_t sb = mira::i4_scale_bits(std::fmax(alpha, eps) / (float)mira::kI4QMax);
        const float sc = mira::i4_scale_value(sb);
        auto q = [&](float v) {
          const float t = std::rint(v / sc);
          return (int)std::fmin(std::fmax(t, -(float)mira::kI4QMax), (float)mira::kI4QMax);
        };
        for (int gq = 0; gq < 4; ++gq) {
          uint8_t* run = m + mira::i4_half_run_offset(r, blk, gq, K);
          for (int bb = 0; bb < 8; ++bb) {
            const int c = 16 * gq + 8 * (bb >> 2) + (bb & 3);
            run[bb] = (uint8_t)(((q(w[c]) & 0xF) << 4) | (q(w[c + 4]) & 0xF));
          }
        }
        std::memcpy(m + mira::i4_scale_offset(r, blk, mat == 2 ? C : R, K), &sb, 2);
      }
    }
  });
  const size_t used = 2 * mira::i4_matrix_bytes(R, C) + mira::i4_matrix_bytes(C, R);
  std::memset(blob + used, 0, stride - used);
}

}  // namespace

namespace mira {

void prof_begin(const char* name, hipStream_t st) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (!g_prof_on) return;
  if (!g_prof_only.empty() && g_prof_only != name) return;
  ProfRec r{name, prof_event(), nullptr};
  if (r.a) (void)hipEventRecord(r.a, st);  // timing only: a failed record drops the sample
  g_prof.push_back(r);
}

void prof_events(const char* name, hipEvent_t* start, hipEvent_t* stop) {
  *start = *stop = nullptr;
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (!g_prof_on) return;
  if (!g_prof_only.empty() && g_prof_only != name) return;
  ProfRec r{name, prof_event(), prof_event()};
  if (!r.a || !r.b) return;
  *start = r.a;
  *stop = r.b;
  g_prof.push_back(r);
}
void prof_end(const char* name, hipStream_t st) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  if (!g_prof_on) return;
  if (!g_prof_only.empty() && g_prof_only != name) return;
  for (auto it = g_prof.rbegin(); it != g_prof.rend(); ++it) {
    if (it->b == nullptr && std::strcmp(it->name, name) == 0) {
      it->b = prof_event();
      if (it->b) (void)hipEventRecord(it->b, st);
      return;
    }
  }
}

int set_error(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int clear_error() { return ok(); }

int device_cu_count() {
  static std::mutex mu;
  static std::map<int, int> cache;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  std::lock_guard<std::mutex> g(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) return it->second;
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  cache[dev] = n;
  return n;
}

}  // namespace mira

extern "C" {

size_t mira_packed_expert_bytes_int4(int32_t hidden, int32_t ffn) {
  if (hidden <= 0 || ffn <= 0 || hidden % 128 || ffn % 128) return 0;
  const unsigned __int128 raw = (unsigned __int128)3 * hidden * ffn * 17 / 32;
  const unsigned __int128 r = (raw + 255) / 256 * 256;
  if (r > (unsigned __int128)SIZE_MAX) return 0;
  return (size_t)r;
}

size_t mira_packed_expert_bytes(int32_t hidden, int32_t ffn) {
  if (hidden <= 0 || ffn <= 0) return 0;
  const unsigned __int128 raw = (unsigned __int128)3 * hidden * ffn + (unsigned __int128)2 * ffn;
  const unsigned __int128 r = (raw + 255) / 256 * 256;
  if (r > (unsigned __int128)SIZE_MAX) return 0;
  return (size_t)r;
}

size_t mira_workspace_bytes(const mira_shape* s, int32_t max_tokens) {
  if (check_shape(s) || max_tokens < 0) return 0;
  return mira::make_layout(*s, max_tokens).total;
}

int mira_pack_experts(const mira_shape* s, int32_t n_experts, int32_t w_dtype, const void* w_gate,
                      const void* w_up, const void* w_down, float eps, void* packed,
                      uint64_t packed_stride, int32_t on_device, hipStream_t stream) {
  if (!s) return fail(MIRA_ERR_ARG, "shape is NULL");
  const int C = s->hidden, R = s->ffn;
  if (C <= 0 || R <= 0) return fail(MIRA_ERR_SHAPE, "hidden and ffn must be positive");
  if (n_experts < 0) return fail(MIRA_ERR_SHAPE, "n_experts must be >= 0");
  if (w_dtype != MIRA_F32 && w_dtype != MIRA_BF16) return fail(MIRA_ERR_ARG, "bad w_dtype");
  if (!(eps > 0.f) || !std::isfinite(eps)) return fail(MIRA_ERR_ARG, "eps must be positive and finite");
  if (on_device != 0 && on_device != 1) return fail(MIRA_ERR_ARG, "on_device must be 0 or 1");
  const bool i4 = s->flags & MIRA_FLAG_INT4;
  if (i4 && (C % 128 || R % 128)) return fail(MIRA_ERR_SHAPE, "INT4 packing needs hidden and ffn multiples of 128");
  const size_t need = i4 ? mira_packed_expert_bytes_int4(C, R) : mira_packed_expert_bytes(C, R);
  if (need == 0) return fail(MIRA_ERR_SHAPE, "expert size overflows");
  if (packed_stride % 256 || packed_stride < need)
    return fail(MIRA_ERR_SHAPE, "packed_stride must be a multiple of 256 and >= %zu", need);
  if (n_experts == 0) return ok();
  if (!w_gate || !w_up || !w_down || !packed) return fail(MIRA_ERR_ARG, "NULL weight or output pointer");
  const size_t esz = w_dtype == MIRA_F32 ? 4 : 2;
  if (on_device) {
    if (!aligned(packed, 256)) return fail(MIRA_ERR_ALIGN, "packed must be 256-byte aligned");
    if (i4)
      HIP_TRY(mira::launch_pack_i4(C, R, n_experts, w_dtype, w_gate, w_up, w_down, eps, packed,
                                   packed_stride, stream));
    else
      HIP_TRY(mira::launch_pack(C, R, n_experts, w_dtype, w_gate, w_up, w_down, eps, packed,
                                packed_stride, stream));
    return ok();
  }
  const size_t per = (size_t)R * C;
  if (i4) {
    for (int e = 0; e < n_experts; ++e) {
      uint8_t* blob = (uint8_t*)packed + (size_t)e * packed_stride;
      if (w_dtype == MIRA_F32)
        host_pack_one_i4<float>(C, R, (const float*)w_gate + e * per, (const float*)w_up + e * per,
                                (const float*)w_down + e * per, eps, blob, packed_stride);
      else
        host_pack_one_i4<uint16_t>(C, R, (const uint16_t*)w_gate + e * per,
                                   (const uint16_t*)w_up + e * per,
                                   (const uint16_t*)w_down + e * per, eps, blob, packed_stride);
    }
    return ok();
  }
  for (int e = 0; e < n_experts; ++e) {
    int8_t* blob = (int8_t*)packed + (size_t)e * packed_stride;
    if (w_dtype == MIRA_F32)
      host_pack_one<float>(C, R, (const float*)w_gate + e * per, (const float*)w_up + e * per,
                           (const float*)w_down + e * per, eps, blob, packed_stride);
    else
      host_pack_one<uint16_t>(C, R, (const uint16_t*)w_gate + e * per,
                              (const uint16_t*)w_up + e * per, (const uint16_t*)w_down + e * per,
                              eps, blob, packed_stride);
  }
  (void)esz;
  return ok();
}

int mira_moe_route(const mira_shape* s, const mira_moe_args* a, hipStream_t stream) {
  mira::Layout L;
  int rc = check_args(s, a, &L);
  if (rc) return rc;
  if (a->n_tokens == 0) return ok();
  rc = run_route(s, a, L, stream);
  return rc ? rc : ok();
}

int mira_moe_experts(const mira_shape* s, const mira_moe_args* a, hipStream_t stream) {
  mira::Layout L;
  int rc = check_args(s, a, &L);
  if (rc) return rc;
  if (a->n_tokens == 0) return ok();
  rc = run_experts(s, a, L, stream);
  return rc ? rc : ok();
}

int mira_moe_forward(const mira_shape* s, const mira_moe_args* a, hipStream_t stream) {
  mira::Layout L;
  int rc = check_args(s, a, &L);
  if (rc) return rc;
  if (a->n_tokens == 0) return ok();
  rc = run_route(s, a, L, stream);
  if (rc) return rc;
  rc = run_experts(s, a, L, stream);
  return rc ? rc : ok();
}

int mira_moe_forward_noalloc(const mira_shape* s, const mira_moe_args* a, hipStream_t stream) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (!a) return fail(MIRA_ERR_ARG, "args is NULL");
  if (a->workspace || a->workspace_bytes)
    return fail(MIRA_ERR_ARG, "the workspace-free call takes workspace = NULL and workspace_bytes = 0");
  if (a->n_tokens < 0) return fail(MIRA_ERR_SHAPE, "n_tokens must be >= 0");
  const size_t need = mira_workspace_bytes(s, a->n_tokens);
  if (need > MIRA_NOALLOC_SCRATCH_BYTES)
    return fail(MIRA_ERR_WORKSPACE,
                "%d tokens need %zu bytes of workspace; the library's scratch holds %u "
                "(MIRA_NOALLOC_SCRATCH_BYTES): use mira_moe_forward with a workspace",
                a->n_tokens, need, (unsigned)MIRA_NOALLOC_SCRATCH_BYTES);
  void* scratch = nullptr;
  HIP_TRY(mira::noalloc_scratch(&scratch));
  mira_moe_args b = *a;
  b.workspace = scratch;
  b.workspace_bytes = MIRA_NOALLOC_SCRATCH_BYTES;
  return mira_moe_forward(s, &b, stream);
}

size_t mira_predict_workspace_bytes(const mira_pred_shape* p, int32_t n_tokens) {
  if (!p || p->group < 1 || p->hidden <= 0 || p->pred_hidden <= 0 || n_tokens < 0) return 0;
  const size_t n = (size_t)(n_tokens / p->group);
  return mira::align_up(n * p->hidden * 4, 256) + mira::align_up(n * p->pred_hidden * 4, 256);
}

int mira_predict(const mira_pred_shape* p, const void* x, int32_t n_tokens, const void* w1,
                 const float* b1, const void* w2, const float* b2, float* scores, void* workspace,
                 uint64_t workspace_bytes, hipStream_t stream) {
  if (!p) return fail(MIRA_ERR_ARG, "pred shape is NULL");
  if (p->reserved != 0) return fail(MIRA_ERR_ARG, "pred shape reserved must be 0");
  if (p->hidden <= 0 || p->hidden % 64) return fail(MIRA_ERR_SHAPE, "hidden must be a positive multiple of 64");
  if (p->pred_hidden < 1) return fail(MIRA_ERR_SHAPE, "pred_hidden must be >= 1");
  if (p->n_out < 1 || p->n_out > MIRA_MAX_EXPERTS) return fail(MIRA_ERR_SHAPE, "n_out out of range");
  if (p->group < 1) return fail(MIRA_ERR_SHAPE, "group must be >= 1");
  if (p->act_dtype != MIRA_F32 && p->act_dtype != MIRA_BF16) return fail(MIRA_ERR_ARG, "bad act_dtype");
  if (n_tokens < 0 || n_tokens % p->group)
    return fail(MIRA_ERR_SHAPE, "n_tokens (%d) must be a non-negative multiple of group (%d)",
                n_tokens, p->group);
  if (n_tokens == 0) return ok();
  if (!x || !w1 || !w2 || !scores || !workspace) return fail(MIRA_ERR_ARG, "NULL pointer argument");
  if (!aligned(w1, 16)) return fail(MIRA_ERR_ALIGN, "w1 must be 16-byte aligned");
  if (!aligned(workspace, 256)) return fail(MIRA_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (workspace_bytes < mira_predict_workspace_bytes(p, n_tokens))
    return fail(MIRA_ERR_WORKSPACE, "predict workspace too small");
  HIP_TRY(mira::launch_predict(*p, x, n_tokens, w1, b1, w2, b2, scores, workspace, stream));
  return ok();
}

size_t mira_mixture_workspace_bytes(const mira_mixture_shape* p, int32_t n_tokens) {
  if (!p || p->group < 1 || p->hidden <= 0 || p->n_src <= 0 || p->act_hidden <= 0 ||
      p->hist_hidden <= 0 || n_tokens < 0)
    return 0;
  return mira::mixture_ws_bytes(n_tokens / p->group, *p);
}

int mira_predict_mixture(const mira_mixture_shape* p, const mira_mixture_weights* w, const void* x,
                         const float* logits, const int32_t* topk_idx, int32_t n_tokens,
                         float* probs, float* alpha, void* workspace, uint64_t workspace_bytes,
                         hipStream_t stream) {
  if (!p || !w) return fail(MIRA_ERR_ARG, "mixture shape or weights is NULL");
  if (p->reserved != 0 || w->reserved != 0) return fail(MIRA_ERR_ARG, "reserved fields must be 0");
  if (p->hidden <= 0 || p->hidden % 64) return fail(MIRA_ERR_SHAPE, "hidden must be a positive multiple of 64");
  if (p->n_src < 1 || p->n_src > MIRA_MAX_EXPERTS) return fail(MIRA_ERR_SHAPE, "n_src out of range");
  if (p->top_k < 1 || p->top_k > MIRA_MAX_TOPK) return fail(MIRA_ERR_SHAPE, "top_k out of range");
  if (p->hist_top < 1 || p->hist_top > p->n_src) return fail(MIRA_ERR_SHAPE, "hist_top must lie in 1..n_src");
  if (p->act_hidden < 1 || p->hist_hidden < 1) return fail(MIRA_ERR_SHAPE, "head widths must be >= 1");
  if (p->n_out < 1 || p->n_out > MIRA_MAX_EXPERTS) return fail(MIRA_ERR_SHAPE, "n_out out of range");
  if (p->group < 1) return fail(MIRA_ERR_SHAPE, "group must be >= 1");
  if (p->act_dtype != MIRA_F32 && p->act_dtype != MIRA_BF16) return fail(MIRA_ERR_ARG, "bad act_dtype");
  if (n_tokens < 0 || n_tokens % p->group)
    return fail(MIRA_ERR_SHAPE, "n_tokens (%d) must be a non-negative multiple of group (%d)",
                n_tokens, p->group);
  if ((int64_t)p->group * p->top_k > INT32_MAX) return fail(MIRA_ERR_SHAPE, "group * top_k overflows");
  if (n_tokens == 0) return ok();
  if (!x || !logits || !topk_idx || !probs || !workspace) return fail(MIRA_ERR_ARG, "NULL pointer argument");
  if (!w->wah || !w->wal || !w->wa2 || !w->whq || !w->whu || !w->wh2 || !w->gh || !w->gl ||
      !w->gq || !w->gu)
    return fail(MIRA_ERR_ARG, "NULL weight pointer");
  if (!aligned(x, 16) || !aligned(w->wah, 16) || !aligned(w->gh, 16))
    return fail(MIRA_ERR_ALIGN, "x, wah and gh must be 16-byte aligned");
  if (!aligned(workspace, 256)) return fail(MIRA_ERR_ALIGN, "workspace must be 256-byte aligned");
  if (workspace_bytes < mira_mixture_workspace_bytes(p, n_tokens))
    return fail(MIRA_ERR_WORKSPACE, "mixture workspace too small");
  HIP_TRY(mira::launch_mixture(*p, *w, x, logits, topk_idx, n_tokens, probs, alpha, workspace, stream));
  return ok();
}

int mira_stage_expert(void* slot_pool, uint64_t slot_stride, int32_t slot, const void* pinned_src,
                      uint64_t bytes, hipStream_t copy_stream, hipEvent_t done) {
  if (!slot_pool || !pinned_src) return fail(MIRA_ERR_ARG, "NULL pool or source");
  if (slot < 0) return fail(MIRA_ERR_ARG, "slot must be >= 0");
  if (bytes > slot_stride) return fail(MIRA_ERR_SHAPE, "bytes exceed slot_stride");
  char* dst = (char*)slot_pool + (size_t)slot * slot_stride;
  mira::prof_begin("stage_copy", copy_stream);
  HIP_TRY(hipMemcpyAsync(dst, pinned_src, bytes, hipMemcpyHostToDevice, copy_stream));
  mira::prof_end("stage_copy", copy_stream);
  if (done) HIP_TRY(hipEventRecord(done, copy_stream));
  return ok();
}

int mira_set_slot(int32_t* slot_table, int32_t expert, int32_t slot, hipStream_t stream) {
  if (!slot_table) return fail(MIRA_ERR_ARG, "slot_table is NULL");
  if (expert < 0 || expert >= MIRA_MAX_EXPERTS) return fail(MIRA_ERR_ARG, "expert out of range");
  if (slot < -1) return fail(MIRA_ERR_ARG, "slot must be >= -1");
  HIP_TRY(mira::launch_set_slot(slot_table, expert, slot, stream));
  return ok();
}

const char* mira_last_error(void) { return g_err.c_str(); }

const char* mira_version(void) { return "mira-mi355x 0.1.0 (gfx950)"; }

int mira_profile_enable(int32_t enable) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  g_prof_on = enable != 0;
  return MIRA_OK;
}

int mira_profile_select(const char* kernel_name) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  g_prof_only = kernel_name ? kernel_name : "";
  return MIRA_OK;
}

int mira_profile_read(int32_t max_entries, const char** names, int32_t* counts, double* total_ms,
                      int32_t* n_entries) {
  std::lock_guard<std::mutex> g(g_prof_mu);
  std::vector<std::pair<const char*, std::pair<int, double>>> agg;
  for (auto& r : g_prof) {
    if (!r.a || !r.b) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) continue;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) continue;
    auto it = std::find_if(agg.begin(), agg.end(),
                           [&](const auto& x) { return std::strcmp(x.first, r.name) == 0; });
    if (it == agg.end()) agg.push_back({r.name, {1, (double)ms}});
    else {
      it->second.first += 1;
      it->second.second += ms;
    }
  }
  for (auto& r : g_prof) {
    if (r.a) g_prof_free.push_back(r.a);
    if (r.b) g_prof_free.push_back(r.b);
  }
  g_prof.clear();
  const int n = (int)agg.size();
  if (n_entries) *n_entries = n;
  for (int i = 0; i < n && i < max_entries; ++i) {
    if (names) names[i] = agg[i].first;
    if (counts) counts[i] = agg[i].second.first;
    if (total_ms) total_ms[i] = agg[i].second.second;
  }
  g_err.clear();
  return MIRA_OK;
}

}  // extern "C"
