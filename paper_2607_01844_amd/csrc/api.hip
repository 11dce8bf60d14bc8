// C ABI of the MoE library: argument validation (pure host code, run before
// any HIP call), workspace queries, status strings and the optional
// per-kernel event profiler.  Kernels live in route/permute/combine/gemm.hip.
#include <atomic>
#include <cstdio>
#include <mutex>
#include <string>
#include <vector>

#include "common.h"

#define MOE_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local std::string g_last_error;

int fail(int status, const char* fn, const char* what) {
  char buf[512];
  std::snprintf(buf, sizeof buf, "%s: %s", fn, what);
  g_last_error = buf;
  return status;
}

int hip_status(hipError_t e, const char* fn) {
  if (e == hipSuccess) return MOE_OK;
  return fail(MOE_ERR_HIP, fn, hipGetErrorString(e));
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

#define REQ(ptr)                                                                   \
  do {                                                                             \
    if ((ptr) == nullptr) return fail(MOE_ERR_INVALID_ARG, fn, #ptr " is NULL");   \
    if (!aligned16(ptr)) return fail(MOE_ERR_INVALID_ARG, fn, #ptr " not 16-byte aligned"); \
  } while (0)
#define OPT(ptr)                                                                   \
  do {                                                                             \
    if ((ptr) != nullptr && !aligned16(ptr))                                       \
      return fail(MOE_ERR_INVALID_ARG, fn, #ptr " not 16-byte aligned");          \
  } while (0)
#define CHECK(cond, msg)                                                           \
  do {                                                                             \
    if (!(cond)) return fail(MOE_ERR_INVALID_ARG, fn, msg);                        \
  } while (0)

int check_tk(const char* fn, int64_t T, int E, int k) {
  CHECK(T >= 0, "T < 0");
  CHECK(E >= 1 && E <= MOE_MAX_E, "E out of [1, MOE_MAX_E]");
  CHECK(k >= 1 && k <= MOE_MAX_K, "k out of [1, MOE_MAX_K]");
  CHECK(k <= E, "k > E");
  CHECK(T * static_cast<int64_t>(k) < (int64_t{1} << 31), "T*k >= 2^31");
  return MOE_OK;
}
int check_dim(const char* fn, int v, const char* name) {
  if (v < 8 || (v % 8) != 0 || v > MOE_MAX_DIM) {
    std::string m = std::string(name) + " must be a multiple of 8 in [8, MOE_MAX_DIM]";
    return fail(MOE_ERR_INVALID_ARG, fn, m.c_str());
  }
  return MOE_OK;
}

// ------------------------------------------------------------ profiler
struct Prof {
  std::mutex mu;
  bool on = false;
  std::vector<std::pair<hipEvent_t, hipEvent_t>> ev[moe::K_NUM];
  std::vector<hipEvent_t> pool;
  hipEvent_t pending[moe::K_NUM] = {};
};
Prof& prof() {
  static Prof p;
  return p;
}
hipEvent_t take_event(Prof& p) {
  if (!p.pool.empty()) {
    hipEvent_t e = p.pool.back();
    p.pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

const char* const kNames[moe::K_NUM] = {
    "route_logits", "route_topk",      "permute_count",      "permute_scan",
    "permute_rank", "permute_gather",  "gemm_sched",         "gemm_fwd_gate_up",
    "gemm_fwd_down", "gemm_dgrad_down", "gemm_dgrad_gate_up", "gemm_wgrad_gate_up",
    "gemm_wgrad_down", "combine",       "combine_bwd",        "route_dlogits",
    "route_dw",     "route_dx",        "vocab_lse",          "vocab_grad",    "llep_plan",     "llep_window",
    "route_split",  "vocab_logits",    "vocab_dx",           "vocab_dw"};

}  // namespace

namespace moe {
int device_cus() {
  constexpr int kMaxDev = 64;
  static std::atomic<int> cache[kMaxDev];
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (dev >= 0 && dev < kMaxDev && (n = cache[dev].load(std::memory_order_relaxed)) > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  if (dev >= 0 && dev < kMaxDev) cache[dev].store(n, std::memory_order_relaxed);
  return n;
}

void prof_begin(int id, hipStream_t s) {
  Prof& p = prof();
  if (!p.on) return;
  std::lock_guard<std::mutex> g(p.mu);
  hipEvent_t e = take_event(p);
  if (e && hipEventRecord(e, s) == hipSuccess) p.pending[id] = e;
}
void prof_end(int id, hipStream_t s) {
  Prof& p = prof();
  if (!p.on) return;
  std::lock_guard<std::mutex> g(p.mu);
  hipEvent_t b = p.pending[id];
  p.pending[id] = nullptr;
  if (!b) return;
  hipEvent_t e = take_event(p);
  if (e && hipEventRecord(e, s) == hipSuccess) p.ev[id].emplace_back(b, e);
}
}  // namespace moe

MOE_API int moe_abi_version(void) { return MOE_ABI_VERSION; }

MOE_API const char* moe_status_string(int status) {
  switch (status) {
    case MOE_OK: return "MOE_OK";
    case MOE_ERR_INVALID_ARG: return "MOE_ERR_INVALID_ARG";
    case MOE_ERR_UNSUPPORTED: return "MOE_ERR_UNSUPPORTED";
    case MOE_ERR_WORKSPACE: return "MOE_ERR_WORKSPACE";
    case MOE_ERR_HIP: return "MOE_ERR_HIP";
    default: return "MOE_ERR_UNKNOWN";
  }
}

MOE_API const char* moe_last_error(void) { return g_last_error.c_str(); }

// ------------------------------------------------------------------ router
MOE_API int moe_route_workspace_bytes(int64_t T, int E, size_t* bytes) {
  const char* fn = "moe_route_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  CHECK(T >= 0 && T < (int64_t{1} << 31), "T out of [0, 2^31)");
  CHECK(E >= 1 && E <= MOE_MAX_E, "E out of [1, MOE_MAX_E]");
  *bytes = moe::align_up(sizeof(float) * static_cast<size_t>(T) * E, 256);
  return MOE_OK;
}

MOE_API int moe_route(const moe_bf16* x, const float* w_router, const float* router_bias,
                      int64_t T, int d, int E, int k, int renorm, int32_t* topk_idx,
                      float* topk_gate, float* logits, void* workspace, size_t workspace_bytes,
                      void* stream) {
  const char* fn = "moe_route";
  if (int r = check_tk(fn, T, E, k)) return r;
  if (int r = check_dim(fn, d, "d")) return r;
  CHECK(renorm == 0 || renorm == 1, "renorm must be 0 or 1");
  if (T > 0) {
    REQ(x); REQ(w_router); REQ(topk_idx); REQ(topk_gate);
    OPT(router_bias); OPT(logits);
  }
  float* lg = logits;
  if (lg == nullptr && T > 0) {
    size_t need = 0;
    moe_route_workspace_bytes(T, E, &need);
    if (workspace == nullptr || workspace_bytes < need)
      return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_route_workspace_bytes()");
    OPT(workspace);
    lg = static_cast<float*>(workspace);
  }
  return hip_status(moe::launch_route(x, w_router, router_bias, T, d, E, k, renorm, topk_idx,
                                      topk_gate, lg, static_cast<hipStream_t>(stream)),
                    fn);
}

MOE_API int moe_route_bwd_workspace_bytes(int64_t T, int d, int E, size_t* bytes) {
  const char* fn = "moe_route_bwd_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  CHECK(T >= 0 && T < (int64_t{1} << 31), "T out of [0, 2^31)");
  CHECK(E >= 1 && E <= MOE_MAX_E, "E out of [1, MOE_MAX_E]");
  if (int r = check_dim(fn, d, "d")) return r;
  *bytes = moe::route_bwd_ws_bytes(T, d, E);
  return MOE_OK;
}

MOE_API int moe_route_bwd(const moe_bf16* x, const float* w_router, const float* logits,
                          const int32_t* topk_idx, const float* topk_gate, const float* dgate,
                          int64_t T, int d, int E, int k, int renorm, float* dw_router,
                          float* dbias, moe_bf16* dx, int dx_accumulate, float* dlogits,
                          void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "moe_route_bwd";
  if (int r = check_tk(fn, T, E, k)) return r;
  if (int r = check_dim(fn, d, "d")) return r;
  CHECK(renorm == 0 || renorm == 1, "renorm must be 0 or 1");
  CHECK(dx_accumulate == 0 || dx_accumulate == 1, "dx_accumulate must be 0 or 1");
  REQ(dw_router);
  OPT(dbias);
  if (T > 0) {
    REQ(x); REQ(w_router); REQ(logits); REQ(topk_idx); REQ(topk_gate); REQ(dgate);
    OPT(dx); OPT(dlogits);
  }
  size_t need = moe::route_bwd_ws_bytes(T, d, E);
  if (dlogits != nullptr) need -= moe::align_up(sizeof(float) * static_cast<size_t>(T) * E, 256);
  if (need > 0) {
    if (workspace == nullptr || workspace_bytes < need)
      return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_route_bwd_workspace_bytes()");
    OPT(workspace);
  }
  return hip_status(moe::launch_route_bwd(x, w_router, logits, topk_idx, topk_gate, dgate, T, d,
                                          E, k, renorm, dw_router, dbias, dx, dx_accumulate,
                                          dlogits, workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------- permutation
MOE_API int moe_permute_workspace_bytes(int64_t T, int E, int k, int num_local, size_t* bytes) {
  const char* fn = "moe_permute_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  if (int r = check_tk(fn, T, E, k)) return r;
  CHECK(num_local >= 1 && num_local <= E, "num_local out of [1, E]");
  *bytes = moe::permute_ws_bytes(T, E, k, num_local);
  return MOE_OK;
}

MOE_API int moe_permute(const moe_bf16* x, const int32_t* topk_idx, int64_t T, int d, int E,
                        int k, int expert_begin, int num_local, int32_t* expert_offsets,
                        int32_t* counts_global, int32_t* row_src, int32_t* dst,
                        moe_bf16* x_perm, void* workspace, size_t workspace_bytes,
                        void* stream) {
  const char* fn = "moe_permute";
  if (int r = check_tk(fn, T, E, k)) return r;
  if (int r = check_dim(fn, d, "d")) return r;
  CHECK(num_local >= 1, "num_local < 1");
  CHECK(expert_begin >= 0 && static_cast<int64_t>(expert_begin) + num_local <= E,
        "expert range outside [0, E)");
  REQ(expert_offsets);
  OPT(counts_global);
  if (T > 0) {
    REQ(x); REQ(topk_idx); REQ(row_src); REQ(dst); REQ(x_perm);
  }
  const size_t need = moe::permute_ws_bytes(T, E, k, num_local);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_permute_workspace_bytes()");
  OPT(workspace);
  return hip_status(moe::launch_permute(x, topk_idx, T, d, E, k, expert_begin, num_local,
                                        expert_offsets, counts_global, row_src, dst, x_perm,
                                        workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

MOE_API int moe_permute_noalloc(const moe_bf16* x, const int32_t* topk_idx, int64_t T, int d,
                                int E, int k, int expert_begin, int num_local,
                                int32_t* expert_offsets, int32_t* counts_global,
                                int32_t* row_src, int32_t* dst, moe_bf16* x_perm, void* stream) {
  const char* fn = "moe_permute_noalloc";
  if (int r = check_tk(fn, T, E, k)) return r;
  if (int r = check_dim(fn, d, "d")) return r;
  CHECK(num_local >= 1, "num_local < 1");
  CHECK(expert_begin >= 0 && static_cast<int64_t>(expert_begin) + num_local <= E,
        "expert range outside [0, E)");
  REQ(expert_offsets);
  OPT(counts_global);
  if (T > 0) {
    REQ(x); REQ(topk_idx); REQ(row_src); REQ(dst); REQ(x_perm);
  }
  if (moe::permute_ws_bytes(T, E, k, num_local) > MOE_PERMUTE_NOALLOC_MAX_BYTES)
    return fail(MOE_ERR_UNSUPPORTED, fn,
                "the scratch this size needs (moe_permute_workspace_bytes) exceeds "
                "MOE_PERMUTE_NOALLOC_MAX_BYTES; use moe_permute with a workspace");
  return hip_status(moe::launch_permute_noalloc(x, topk_idx, T, d, E, k, expert_begin, num_local,
                                                expert_offsets, counts_global, row_src, dst,
                                                x_perm, static_cast<hipStream_t>(stream)),
                    fn);
}

// ----------------------------------------------------- grouped SwiGLU FFN
MOE_API int moe_grouped_swiglu_workspace_bytes(int64_t cap, int num_local, int d, int f,
                                               unsigned flags, size_t* bytes) {
  const char* fn = "moe_grouped_swiglu_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  CHECK(cap >= 0 && cap < (int64_t{1} << 31), "cap out of [0, 2^31)");
  CHECK(num_local >= 1 && num_local <= MOE_MAX_E, "num_local out of [1, MOE_MAX_E]");
  if (int r = check_dim(fn, d, "d")) return r;
  if (int r = check_dim(fn, f, "f")) return r;
  CHECK((flags & ~3u) == 0, "unknown flags");
  *bytes = moe::gemm_ws_bytes(cap, num_local, d, f, flags);
  return MOE_OK;
}

static int check_ffn(const char* fn, int num_local, int64_t cap, int d, int f) {
  CHECK(num_local >= 1 && num_local <= MOE_MAX_E, "num_local out of [1, MOE_MAX_E]");
  CHECK(cap >= 0 && cap < (int64_t{1} << 31), "cap out of [0, 2^31)");
  if (int r = check_dim(fn, d, "d")) return r;
  if (int r = check_dim(fn, f, "f")) return r;
  CHECK(static_cast<int64_t>(d) * f < (int64_t{1} << 31), "d*f >= 2^31");
  CHECK(cap * std::max(d, f) < (int64_t{1} << 40), "cap*max(d,f) too large");
  return MOE_OK;
}

MOE_API int moe_grouped_swiglu_fwd(const moe_bf16* x_perm, const int32_t* expert_offsets,
                                   int num_local, int64_t cap, int d, int f,
                                   const moe_bf16* w_gate, const moe_bf16* w_up,
                                   const moe_bf16* w_down, moe_bf16* h_gate, moe_bf16* h_up,
                                   moe_bf16* y_perm, void* workspace, size_t workspace_bytes,
                                   void* stream) {
  const char* fn = "moe_grouped_swiglu_fwd";
  if (int r = check_ffn(fn, num_local, cap, d, f)) return r;
  REQ(expert_offsets); REQ(w_gate); REQ(w_up); REQ(w_down);
  if (cap > 0) {
    REQ(x_perm); REQ(h_gate); REQ(h_up); REQ(y_perm);
  }
  const size_t need = moe::gemm_ws_bytes(cap, num_local, d, f, 0);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_grouped_swiglu_workspace_bytes()");
  OPT(workspace);
  return hip_status(moe::launch_ffn_fwd(x_perm, expert_offsets, num_local, cap, d, f, w_gate,
                                        w_up, w_down, h_gate, h_up, y_perm, workspace,
                                        static_cast<hipStream_t>(stream)),
                    fn);
}

MOE_API int moe_grouped_swiglu_bwd(const moe_bf16* dy_perm, const moe_bf16* x_perm,
                                   const moe_bf16* h_gate, const moe_bf16* h_up,
                                   const int32_t* expert_offsets, int num_local, int64_t cap,
                                   int d, int f, const moe_bf16* w_gate, const moe_bf16* w_up,
                                   const moe_bf16* w_down, moe_bf16* dx_perm, moe_bf16* dw_gate,
                                   moe_bf16* dw_up, moe_bf16* dw_down, unsigned flags,
                                   void* workspace, size_t workspace_bytes, void* stream) {
  const char* fn = "moe_grouped_swiglu_bwd";
  if (int r = check_ffn(fn, num_local, cap, d, f)) return r;
  CHECK(flags != 0 && (flags & ~3u) == 0, "flags must be a non-empty subset of DGRAD|WGRAD");
  REQ(expert_offsets); REQ(w_down);
  if (cap > 0) {
    REQ(dy_perm); REQ(h_gate); REQ(h_up);
  }
  if (flags & MOE_BWD_DGRAD) {
    REQ(w_gate); REQ(w_up);
    if (cap > 0) REQ(dx_perm);
  }
  if (flags & MOE_BWD_WGRAD) {
    REQ(dw_gate); REQ(dw_up); REQ(dw_down);
    if (cap > 0) REQ(x_perm);
  }
  const size_t need = moe::gemm_ws_bytes(cap, num_local, d, f, flags);
  if (workspace == nullptr || workspace_bytes < need)
    return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_grouped_swiglu_workspace_bytes()");
  OPT(workspace);
  return hip_status(moe::launch_ffn_bwd(dy_perm, x_perm, h_gate, h_up, expert_offsets, num_local,
                                        cap, d, f, w_gate, w_up, w_down, dx_perm, dw_gate,
                                        dw_up, dw_down, flags, workspace,
                                        static_cast<hipStream_t>(stream)),
                    fn);
}

// ----------------------------------------------------------------- combine
MOE_API int moe_combine(const moe_bf16* y_perm, const int32_t* dst, const float* topk_gate,
                        int64_t T, int d, int k, moe_bf16* out, void* stream) {
  const char* fn = "moe_combine";
  CHECK(T >= 0, "T < 0");
  CHECK(k >= 1 && k <= MOE_MAX_K, "k out of [1, MOE_MAX_K]");
  CHECK(T * static_cast<int64_t>(k) < (int64_t{1} << 31), "T*k >= 2^31");
  if (int r = check_dim(fn, d, "d")) return r;
  if (T > 0) {
    REQ(y_perm); REQ(dst); REQ(out);
    OPT(topk_gate);
  }
  return hip_status(moe::launch_combine(y_perm, dst, topk_gate, T, d, k, out,
                                        static_cast<hipStream_t>(stream)),
                    fn);
}

MOE_API int moe_combine_bwd(const moe_bf16* dout, const moe_bf16* y_perm, const int32_t* dst,
                            const float* topk_gate, int64_t T, int d, int k, moe_bf16* dy_perm,
                            float* dgate, void* stream) {
  const char* fn = "moe_combine_bwd";
  CHECK(T >= 0, "T < 0");
  CHECK(k >= 1 && k <= MOE_MAX_K, "k out of [1, MOE_MAX_K]");
  CHECK(T * static_cast<int64_t>(k) < (int64_t{1} << 31), "T*k >= 2^31");
  if (int r = check_dim(fn, d, "d")) return r;
  if (T > 0) {
    REQ(dout); REQ(y_perm); REQ(dst); REQ(dy_perm);
    OPT(topk_gate); OPT(dgate);
  }
  return hip_status(moe::launch_combine_bwd(dout, y_perm, dst, topk_gate, T, d, k, dy_perm, dgate,
                                            static_cast<hipStream_t>(stream)),
                    fn);
}

// -------------------------------------------------- memory-efficient forward
MOE_API int moe_ffn_fwd_chunked_workspace_bytes(int64_t chunk, int E, int k, int num_local,
                                                int d, int f, size_t* bytes) {
  const char* fn = "moe_ffn_fwd_chunked_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  CHECK(chunk >= 1, "chunk < 1");
  if (int r = check_tk(fn, chunk, E, k)) return r;
  CHECK(num_local >= 1 && num_local <= E, "num_local out of [1, E]");
  if (int r = check_dim(fn, d, "d")) return r;
  if (int r = check_dim(fn, f, "f")) return r;
  *bytes = moe::ffn_fwd_chunked_ws_bytes(chunk, E, k, num_local, d, f);
  return MOE_OK;
}

MOE_API int moe_ffn_fwd_chunked(const moe_bf16* x, const int32_t* topk_idx, const float* topk_gate,
                                int64_t T, int d, int E, int k, int expert_begin, int num_local,
                                int f, const moe_bf16* w_gate, const moe_bf16* w_up,
                                const moe_bf16* w_down, int64_t chunk, moe_bf16* y,
                                void* workspace, size_t workspace_bytes, void* stream,
                                void* stream2) {
  const char* fn = "moe_ffn_fwd_chunked";
  if (int r = check_tk(fn, T, E, k)) return r;
  CHECK(chunk >= 1, "chunk < 1");
  CHECK(chunk * static_cast<int64_t>(k) < (int64_t{1} << 31), "chunk*k >= 2^31");
  CHECK(num_local >= 1 && num_local <= E, "num_local out of [1, E]");
  CHECK(expert_begin >= 0 && expert_begin + num_local <= E, "expert range out of [0, E)");
  if (int r = check_ffn(fn, num_local, chunk * std::min(k, num_local), d, f)) return r;
  if (T > 0) {
    REQ(x); REQ(topk_idx); REQ(topk_gate); REQ(y);
    REQ(w_gate); REQ(w_up); REQ(w_down);
    const size_t need = moe::ffn_fwd_chunked_ws_bytes(chunk, E, k, num_local, d, f);
    if (workspace == nullptr || workspace_bytes < need)
      return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_ffn_fwd_chunked_workspace_bytes()");
    OPT(workspace);
  }
  return hip_status(moe::launch_ffn_fwd_chunked(x, topk_idx, topk_gate, T, d, E, k, expert_begin,
                                                num_local, f, w_gate, w_up, w_down, chunk, y,
                                                workspace, static_cast<hipStream_t>(stream),
                                                static_cast<hipStream_t>(stream2)),
                    fn);
}

MOE_API int moe_ffn_fwd_row_chunked_workspace_bytes(int64_t T, int E, int k, int num_local,
                                                    int d, int f, int64_t chunk_rows,
                                                    size_t* bytes) {
  const char* fn = "moe_ffn_fwd_row_chunked_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  if (int r = check_tk(fn, T, E, k)) return r;
  CHECK(num_local >= 1 && num_local <= E, "num_local out of [1, E]");
  CHECK(chunk_rows >= 1, "chunk_rows < 1");
  if (int r = check_ffn(fn, num_local, T * std::min(k, num_local), d, f)) return r;
  *bytes = moe::ffn_fwd_row_chunked_ws_bytes(T, E, k, num_local, d, f, chunk_rows);
  return MOE_OK;
}

MOE_API int moe_ffn_fwd_row_chunked(const moe_bf16* x, const int32_t* topk_idx,
                                    const float* topk_gate, int64_t T, int d, int E, int k,
                                    int expert_begin, int num_local, int f,
                                    const moe_bf16* w_gate, const moe_bf16* w_up,
                                    const moe_bf16* w_down, int64_t chunk_rows, moe_bf16* y,
                                    void* workspace, size_t workspace_bytes, void* stream,
                                    void* stream2) {
  const char* fn = "moe_ffn_fwd_row_chunked";
  if (int r = check_tk(fn, T, E, k)) return r;
  CHECK(chunk_rows >= 1, "chunk_rows < 1");
  CHECK(num_local >= 1 && num_local <= E, "num_local out of [1, E]");
  CHECK(expert_begin >= 0 && expert_begin + num_local <= E, "expert range out of [0, E)");
  if (int r = check_ffn(fn, num_local, T * std::min(k, num_local), d, f)) return r;
  if (T > 0) {
    REQ(x); REQ(topk_idx); REQ(topk_gate); REQ(y);
    REQ(w_gate); REQ(w_up); REQ(w_down);
    const size_t need = moe::ffn_fwd_row_chunked_ws_bytes(T, E, k, num_local, d, f, chunk_rows);
    if (workspace == nullptr || workspace_bytes < need)
      return fail(MOE_ERR_WORKSPACE, fn,
                  "workspace smaller than moe_ffn_fwd_row_chunked_workspace_bytes()");
    OPT(workspace);
  }
  return hip_status(moe::launch_ffn_fwd_row_chunked(x, topk_idx, topk_gate, T, d, E, k,
                                                    expert_begin, num_local, f, w_gate, w_up,
                                                    w_down, chunk_rows, y, workspace,
                                                    static_cast<hipStream_t>(stream),
                                                    static_cast<hipStream_t>(stream2)),
                    fn);
}

// ------------------------------------------------------ vocabulary loss
static int check_vocab(const char* fn, int64_t N, int H, int64_t V, int64_t vblock) {
  CHECK(N >= 0 && N < (int64_t{1} << 31), "N out of [0, 2^31)");
  if (int r = check_dim(fn, H, "H")) return r;
  CHECK(V >= 1 && V < (int64_t{1} << 31), "V out of [1, 2^31)");
  CHECK(vblock >= 8 && (vblock % 8) == 0, "vblock must be a positive multiple of 8");
  CHECK(N * vblock < (int64_t{1} << 40), "N*vblock too large");
  return MOE_OK;
}

MOE_API int moe_vocab_loss_workspace_bytes(int64_t N, int H, int64_t V, int64_t vblock,
                                           size_t* bytes) {
  const char* fn = "moe_vocab_loss_workspace_bytes";
  CHECK(bytes != nullptr, "bytes is NULL");
  if (int r = check_vocab(fn, N, H, V, vblock)) return r;
  *bytes = std::max(moe::vocab_fwd_ws_bytes(N, H, V, vblock),
                    moe::vocab_bwd_ws_bytes(N, H, V, vblock));
  return MOE_OK;
}

MOE_API int moe_vocab_loss_fwd(const moe_bf16* x, const moe_bf16* w_voc, const int32_t* target,
                               int64_t N, int H, int64_t V, int64_t vblock, float* loss,
                               float* lse, void* workspace, size_t workspace_bytes,
                               void* stream) {
  const char* fn = "moe_vocab_loss_fwd";
  if (int r = check_vocab(fn, N, H, V, vblock)) return r;
  if (N > 0) {
    REQ(x); REQ(w_voc); REQ(target); REQ(loss); REQ(lse);
    if (workspace == nullptr || workspace_bytes < moe::vocab_fwd_ws_bytes(N, H, V, vblock))
      return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_vocab_loss_workspace_bytes()");
    OPT(workspace);
  }
  return hip_status(moe::launch_vocab_fwd(x, w_voc, target, N, H, V, vblock, loss, lse,
                                          workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

MOE_API int moe_vocab_loss_bwd(const moe_bf16* x, const moe_bf16* w_voc, const int32_t* target,
                               const float* lse, const float* dloss, int64_t N, int H, int64_t V,
                               int64_t vblock, moe_bf16* dx, moe_bf16* dw_voc, void* workspace,
                               size_t workspace_bytes, void* stream) {
  const char* fn = "moe_vocab_loss_bwd";
  if (int r = check_vocab(fn, N, H, V, vblock)) return r;
  REQ(dw_voc);
  if (N > 0) {
    REQ(x); REQ(w_voc); REQ(target); REQ(lse); REQ(dloss); REQ(dx);
    if (workspace == nullptr || workspace_bytes < moe::vocab_bwd_ws_bytes(N, H, V, vblock))
      return fail(MOE_ERR_WORKSPACE, fn, "workspace smaller than moe_vocab_loss_workspace_bytes()");
    OPT(workspace);
  }
  return hip_status(moe::launch_vocab_bwd(x, w_voc, target, lse, dloss, N, H, V, vblock, dx,
                                          dw_voc, workspace, static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------ least-loaded expert parallelism
MOE_API int moe_llep_plan(const int32_t* counts, int E, int E_p, int capacity, int granule,
                          int32_t* win_lo, int32_t* win_hi, int32_t* load, int32_t* n_ship,
                          void* stream) {
  const char* fn = "moe_llep_plan";
  CHECK(E >= 1 && E <= MOE_MAX_E, "E out of [1, MOE_MAX_E]");
  CHECK(E_p >= 1 && E_p <= MOE_LLEP_MAX_RANKS, "E_p out of [1, MOE_LLEP_MAX_RANKS]");
  CHECK(E % E_p == 0, "E must be a multiple of E_p");
  CHECK(capacity >= 0, "capacity < 0");
  CHECK(granule >= 1 && granule <= MOE_LLEP_MAX_GRANULE, "granule out of [1, MOE_LLEP_MAX_GRANULE]");
  REQ(counts); REQ(win_lo); REQ(win_hi); REQ(load); REQ(n_ship);
  return hip_status(moe::launch_llep_plan(counts, E, E_p, capacity, granule, win_lo, win_hi, load,
                                          n_ship, static_cast<hipStream_t>(stream)),
                    fn);
}

MOE_API int moe_llep_dispatch(const moe_bf16* x, const int32_t* topk_idx,
                              const int32_t* offsets_all, const int32_t* dst_all,
                              const int32_t* win_lo, const int32_t* win_hi, int E_p, int rank,
                              int64_t T, int d, int E, int k, int64_t cap, int32_t* offsets_r,
                              int32_t* row_src_r, int32_t* dst_r, moe_bf16* x_perm_r,
                              void* stream) {
  const char* fn = "moe_llep_dispatch";
  if (int r = check_tk(fn, T, E, k)) return r;
  if (int r = check_dim(fn, d, "d")) return r;
  CHECK(E_p >= 1 && E_p <= MOE_LLEP_MAX_RANKS && E % E_p == 0,
        "E_p out of [1, MOE_LLEP_MAX_RANKS] or not a divisor of E");
  CHECK(rank >= 0 && rank < E_p, "rank out of [0, E_p)");
  CHECK(cap >= 0 && cap <= T * k, "cap out of [0, T*k]");
  REQ(offsets_all); REQ(win_lo); REQ(win_hi); REQ(offsets_r);
  if (T > 0) {
    REQ(x); REQ(topk_idx); REQ(dst_all); REQ(dst_r);
    if (cap > 0) { REQ(row_src_r); REQ(x_perm_r); }
  }
  const int64_t o = static_cast<int64_t>(rank) * E;
  return hip_status(moe::launch_llep_dispatch(x, topk_idx, offsets_all, dst_all, win_lo + o,
                                              win_hi + o, T, d, E, k, cap, offsets_r, row_src_r,
                                              dst_r, x_perm_r, static_cast<hipStream_t>(stream)),
                    fn);
}

// ------------------------------------------------------------- profiling
MOE_API int moe_profile_enable(int on) {
  Prof& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  p.on = (on != 0);
  return MOE_OK;
}

MOE_API int moe_profile_reset(void) {
  Prof& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  for (auto& v : p.ev) {
    for (auto& pr : v) {
      p.pool.push_back(pr.first);
      p.pool.push_back(pr.second);
    }
    v.clear();
  }
  return MOE_OK;
}

MOE_API int moe_profile_num_kernels(void) { return moe::K_NUM; }

MOE_API const char* moe_profile_kernel_name(int id) {
  if (id < 0 || id >= moe::K_NUM) return "";
  return kNames[id];
}

MOE_API int moe_profile_query(int id, double* total_ms, int64_t* launches) {
  const char* fn = "moe_profile_query";
  CHECK(id >= 0 && id < moe::K_NUM, "kernel id out of range");
  CHECK(total_ms != nullptr && launches != nullptr, "NULL output");
  Prof& p = prof();
  std::lock_guard<std::mutex> g(p.mu);
  double tot = 0.0;
  for (auto& pr : p.ev[id]) {
    if (hipError_t e = hipEventSynchronize(pr.second); e != hipSuccess) return hip_status(e, fn);
    float ms = 0.0f;
    if (hipError_t e = hipEventElapsedTime(&ms, pr.first, pr.second); e != hipSuccess)
      return hip_status(e, fn);
    tot += ms;
  }
  *total_ms = tot;
  *launches = static_cast<int64_t>(p.ev[id].size());
  return MOE_OK;
}
