// Internal helpers shared by the HIP kernels of the MoE library (gfx950).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

#include "moe.h"

namespace moe {

constexpr int kWave = 64;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------ bf16 helpers
__device__ __forceinline__ float bf16_lo(uint32_t v) { return __uint_as_float(v << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t v) { return __uint_as_float(v & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t v) {
  return __uint_as_float(static_cast<uint32_t>(v) << 16);
}

// fp32 -> bf16, round to nearest even, NaN -> quiet NaN: gfx950's packed
// convert (v_cvt_pk_bf16_f32).  It agrees bit for bit with the integer
// rounding (u + 0x7fff + ((u >> 16) & 1)) >> 16 on every finite input, and
// with (u >> 16) | 0x40 on NaN (checked over all 2^32 fp32 patterns).
typedef __bf16 bf16x2_hw __attribute__((ext_vector_type(2)));
typedef float f32x2_hw __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_hw{lo, hi}, bf16x2_hw));
}
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) { return pack_bf16x2(f, 0.0f) & 0xffffu; }

// ------------------------------------------------------------ wave helpers
__device__ __forceinline__ int lane_id() { return __lane_id(); }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, kWave);
  return v;
}

// Compile-time loop: f(std::integral_constant<int, 0..N-1>) (keeps register
// arrays indexed by constants, so they never fall back to scratch memory).
template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
  (f(std::integral_constant<int, Is>{}), ...);
}
template <int N, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

// ------------------------------------------------------------ math helpers
__device__ __forceinline__ float sigmoidf_fast(float z) { return 1.0f / (1.0f + __expf(-z)); }

// --------------------------------------------------------- launch plumbing
struct LaunchCtx {
  hipStream_t stream;
};

// Kernel ids for the optional profiler (order = moe_profile_kernel_name).
enum KernelId {
  K_ROUTE_LOGITS = 0,
  K_ROUTE_TOPK,
  K_PERM_COUNT,
  K_PERM_SCAN,
  K_PERM_RANK,
  K_PERM_GATHER,
  K_GEMM_SCHED,
  K_GEMM_FWD_GATE_UP,
  K_GEMM_FWD_DOWN,
  K_GEMM_DGRAD_DOWN,
  K_GEMM_DGRAD_GATE_UP,
  K_GEMM_WGRAD_GATE_UP,
  K_GEMM_WGRAD_DOWN,
  K_COMBINE,
  K_COMBINE_BWD,
  K_ROUTE_DLOGITS,
  K_ROUTE_DW,
  K_ROUTE_DX,
  K_VOC_LSE,
  K_VOC_GRAD,
  K_LLEP_PLAN,
  K_LLEP_WINDOW,
  K_ROUTE_SPLIT,
  K_VOC_LOGITS,
  K_VOC_DX,
  K_VOC_DW,
  K_NUM
};

// Profiler hooks (no-ops unless moe_profile_enable(1) was called).
void prof_begin(int id, hipStream_t s);
void prof_end(int id, hipStream_t s);

// Compute units of the current device (cached per device; 256 if the
// query fails).
int device_cus();

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
inline size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

// ------------------------------------------------------ kernel launchers
// (defined next to their kernels; arguments were validated by the C ABI)
hipError_t launch_route(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                        int E, int k, int renorm, int32_t* idx, float* gate, float* logits,
                        hipStream_t s);
int route_bwd_chunks(int64_t T, int d, int E);
size_t route_bwd_ws_bytes(int64_t T, int d, int E);
hipError_t launch_route_bwd(const uint16_t* x, const float* w, const float* logits,
                            const int32_t* idx, const float* gate, const float* dgate,
                            int64_t T, int d, int E, int k, int renorm, float* dw, float* dbias,
                            uint16_t* dx, int dx_accumulate, float* dlogits, void* ws,
                            hipStream_t s);
size_t vocab_fwd_ws_bytes(int64_t N, int H, int64_t V, int64_t vblock);
size_t vocab_bwd_ws_bytes(int64_t N, int H, int64_t V, int64_t vblock);
hipError_t launch_vocab_fwd(const uint16_t* x, const uint16_t* w, const int32_t* target,
                            int64_t N, int H, int64_t V, int64_t vblock, float* loss, float* lse,
                            void* ws, hipStream_t s);
hipError_t launch_vocab_bwd(const uint16_t* x, const uint16_t* w, const int32_t* target,
                            const float* lse, const float* dloss, int64_t N, int H, int64_t V,
                            int64_t vblock, uint16_t* dx, uint16_t* dw, void* ws, hipStream_t s);
size_t ffn_fwd_chunked_ws_bytes(int64_t chunk, int E, int k, int E_loc, int d, int f);
size_t ffn_fwd_row_chunked_ws_bytes(int64_t T, int E, int k, int E_loc, int d, int f,
                                    int64_t chunk_rows);
hipError_t launch_ffn_fwd_row_chunked(const uint16_t* x, const int32_t* idx, const float* gate,
                                      int64_t T, int d, int E, int k, int e_begin, int E_loc,
                                      int f, const uint16_t* wg, const uint16_t* wu,
                                      const uint16_t* wd, int64_t chunk_rows, uint16_t* y,
                                      void* ws, hipStream_t s0, hipStream_t s1);
hipError_t launch_ffn_fwd_chunked(const uint16_t* x, const int32_t* idx, const float* gate,
                                  int64_t T, int d, int E, int k, int e_begin, int E_loc, int f,
                                  const uint16_t* wg, const uint16_t* wu, const uint16_t* wd,
                                  int64_t chunk, uint16_t* y, void* ws, hipStream_t s0,
                                  hipStream_t s1);
size_t permute_ws_bytes(int64_t T, int E, int k, int E_loc);
hipError_t launch_permute(const uint16_t* x, const int32_t* idx, int64_t T, int d, int E, int k,
                          int e_begin, int E_loc, int32_t* offsets, int32_t* counts_global,
                          int32_t* row_src, int32_t* dst, uint16_t* x_perm, void* ws,
                          hipStream_t s);
hipError_t launch_gather(const uint16_t* x, const int32_t* dst, int64_t T, int d, int k,
                         uint16_t* x_perm, hipStream_t s);
// Rows [r0, r0 + rc) of a permutation (offsets, row_src over all local
// experts) as a chunk: offsets_c [E_loc + 1] relative to r0 and clamped to
// [0, rc], and x_perm_c [rc][d] (its filled rows) gathered from x.
hipError_t launch_chunk_rows(const uint16_t* x, const int32_t* row_src, const int32_t* offsets,
                             int E_loc, int64_t r0, int64_t rc, int d, int k, int32_t* offsets_c,
                             uint16_t* x_perm_c, hipStream_t s);
// launch_permute with the library's static scratch as the workspace
// (permute_ws_bytes(T, E, k, E_loc) <= MOE_PERMUTE_NOALLOC_MAX_BYTES, checked
// by the caller)
hipError_t launch_permute_noalloc(const uint16_t* x, const int32_t* idx, int64_t T, int d, int E,
                                  int k, int e_begin, int E_loc, int32_t* offsets,
                                  int32_t* counts_global, int32_t* row_src, int32_t* dst,
                                  uint16_t* x_perm, hipStream_t s);
hipError_t launch_llep_plan(const int32_t* counts, int E, int E_p, int capacity, int granule,
                            int32_t* lo, int32_t* hi, int32_t* load, int32_t* n_ship, hipStream_t s);
hipError_t launch_llep_dispatch(const uint16_t* x, const int32_t* idx, const int32_t* offsets_all,
                                const int32_t* dst_all, const int32_t* lo, const int32_t* hi,
                                int64_t T, int d, int E, int k, int64_t cap, int32_t* offsets_r,
                                int32_t* row_src_r, int32_t* dst_r, uint16_t* x_perm_r,
                                hipStream_t s);
hipError_t launch_combine(const uint16_t* y, const int32_t* dst, const float* gate, int64_t T,
                          int d, int k, uint16_t* out, hipStream_t s);
hipError_t launch_combine_bwd(const uint16_t* dout, const uint16_t* y, const int32_t* dst,
                              const float* gate, int64_t T, int d, int k, uint16_t* dy_perm,
                              float* dgate, hipStream_t s);
size_t gemm_ws_bytes(int64_t cap, int E_loc, int d, int f, unsigned flags);
// Dense products on the grouped GEMM kernel (bf16 operands, fp32 accumulation).
// Router backward, fp32 operands split as bf16 hi + lo: dl3 [T][ld3] holds
// [hi | hi | lo] of the logit gradients (E columns each), w3 [3E][d] holds
// [hi; lo; hi] of W_r^T.
//   part[c][j][e] = sum over tokens t of chunk c of x[t][j] (hi + lo)[t][e]
//   dx[t][j] = bf16([float(dx[t][j]) +] sum over the 3E columns of dl3 w3)
hipError_t launch_router_dw_mfma(const uint16_t* x, const uint16_t* dl3, int64_t T, int d, int E,
                                 int64_t ld3, int64_t chunk, float* part, hipStream_t s);
hipError_t launch_router_dx_mfma(const uint16_t* dl3, const uint16_t* w3, int64_t T, int d, int E,
                                 int64_t ld3, int accumulate, uint16_t* dx, hipStream_t s);
// Vocabulary block [v0, v0 + vb) of W [H][ldw] (B read from column bc0):
//   logits: part[n][c / 64] = (max, sum exp(y - max)) over the block's
//     columns c..c+63 of row n, yt[n] = y[n][target[n] - v0] where the
//     target lies in the block;
//   grad: G[n][c] = bf16(dloss[n] ([v0 + c == target[n]] - exp(y - lse[n]))),
//     zeros for c in [vb, gp);
//   dx: dxa[b][n][h] (=, first) or (+=) sum over c in batch b's kspan
//     columns of G[n][c] W[h][bc0 + c];
//   dw: dw[h][cc0 + c] = bf16(sum_n x[n][h] G[n][c]), row pitch ldd.
hipError_t launch_vocab_logits_mfma(const uint16_t* x, const uint16_t* w, int64_t ldw, int64_t bc0,
                                    int64_t v0, int N, int H, int vb, const int32_t* target,
                                    float* part, float* yt, hipStream_t s);
hipError_t launch_vocab_grad_mfma(const uint16_t* x, const uint16_t* w, int64_t ldw, int64_t bc0,
                                  int64_t v0, int N, int H, int vb, const int32_t* target,
                                  const float* lse, const float* dloss, uint16_t* G, int64_t gp,
                                  hipStream_t s);
hipError_t launch_vocab_dx_mfma(const uint16_t* G, int64_t gp, const uint16_t* w, int64_t ldw,
                                int64_t bc0, int N, int H, int vb, int kspan, int first,
                                float* dxa, hipStream_t s);
hipError_t launch_vocab_dw_mfma(const uint16_t* x, const uint16_t* G, int64_t gp, int N, int H,
                                int vb, uint16_t* dw, int64_t ldd, int64_t cc0, hipStream_t s);
hipError_t launch_ffn_fwd(const uint16_t* x_perm, const int32_t* offsets, int E_loc, int64_t cap,
                          int d, int f, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, uint16_t* hg, uint16_t* hu, uint16_t* y,
                          void* ws, hipStream_t s);
hipError_t launch_ffn_bwd(const uint16_t* dy, const uint16_t* x_perm, const uint16_t* hg,
                          const uint16_t* hu, const int32_t* offsets, int E_loc, int64_t cap,
                          int d, int f, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, uint16_t* dx, uint16_t* dwg, uint16_t* dwu,
                          uint16_t* dwd, unsigned flags, void* ws, hipStream_t s);

}  // namespace moe
