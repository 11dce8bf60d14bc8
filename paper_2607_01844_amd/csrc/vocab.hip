// Blockwise vocabulary projection loss (the MoP paper's data-tensor-parallel
// projection, Sec. 3.4 eq. voc-fwd-loss, on one device: P = 1, blocks of the
// vocabulary instead of ranks).  Y = X W_voc is never written anywhere:
//  * forward, per block of `vblock` columns: one bf16 matrix-core product
//    whose epilogue reduces each row's logits to a (max, sum exp(y - max))
//    pair per 64 columns and picks up the target's logit; a one-wave-per-row
//    kernel merges the block's pairs, in column order, into the row's running
//    pair (blocks in order, so the result repeats bit for bit);
//  * backward, per block: the product is recomputed and its epilogue turns
//    each logit into the logit gradient G = dl ([v == t] - exp(y - lse)),
//    rounded to bf16 (the only per-block buffer, N x vblock bf16); then
//    dX += G W_block^T (fp32, the block's columns cut into K ranges that
//    accumulate into separate fp32 slabs so the product fills the chip) and
//    dW[:, block] = X^T G (bf16, each column written once).
// All products run on the library's grouped GEMM kernel (dense modes).  When
// V is not a multiple of 8 the rows of W and dW are not 16-byte aligned, so
// each block of W is first copied into a padded buffer (and dW's block goes
// through one on the way out).
#include "common.h"

#include <algorithm>

namespace moe {
namespace {

// Merge of two (max, sum of exp(y - max)) pairs; an empty pair is (-inf, 0).
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -__builtin_huge_valf()) return;  // both empty
  s = s * __expf(m - mm) + s2 * __expf(m2 - mm);
  m = mm;
}

// One wave per row n: the block's ng partial pairs part[n][0..ng) merged in
// order (lane l takes groups l, l + 64, ... ascending, then a fixed xor
// tree over the lanes), then merged into the row's running pair (m, s).
__global__ __launch_bounds__(256) void voc_merge_kernel(const float2* __restrict__ part, int ng,
                                                        int64_t N, float* __restrict__ m,
                                                        float* __restrict__ s, int first) {
  const int64_t n = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (n >= N) return;
  const float2* row = part + n * ng;
  float tm = -__builtin_huge_valf(), ts = 0.0f;
  for (int c = lane; c < ng; c += 64) {
    const float2 p = row[c];
    lse_merge(tm, ts, p.x, p.y);
  }
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const float m2 = __shfl_xor(tm, o, 64), s2 = __shfl_xor(ts, o, 64);
    // both lanes of a pair compute the same merge in the same operand order
    if (lane & o) {
      float a = m2, b = s2;
      lse_merge(a, b, tm, ts);
      tm = a;
      ts = b;
    } else {
      lse_merge(tm, ts, m2, s2);
    }
  }
  if (lane == 0) {
    if (first) {
      m[n] = tm;
      s[n] = ts;
    } else {
      float rm = m[n], rs = s[n];
      lse_merge(rm, rs, tm, ts);
      m[n] = rm;
      s[n] = rs;
    }
  }
}

// loss_n = y_{n, t_n} - lse_n, lse_n = m_n + log s_n
__global__ __launch_bounds__(256) void voc_finalize_kernel(const float* __restrict__ m,
                                                           const float* __restrict__ s,
                                                           const float* __restrict__ yt, int64_t N,
                                                           float* __restrict__ loss,
                                                           float* __restrict__ lse) {
  const int64_t n = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (n >= N) return;
  const float l = m[n] + logf(s[n]);
  lse[n] = l;
  loss[n] = yt[n] - l;
}

// dx[i] = bf16(sum over slabs b ascending of dxa[b][i]), 8 values per thread
__global__ __launch_bounds__(256) void voc_dx_sum_kernel(const float* __restrict__ dxa, int slabs,
                                                         int64_t n, uint16_t* __restrict__ dx) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 8;
  if (i >= n) return;  // n = N H is a multiple of 8
  float v[8];
  {
    const float4 a = *reinterpret_cast<const float4*>(dxa + i);
    const float4 b = *reinterpret_cast<const float4*>(dxa + i + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w; v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
  for (int sl = 1; sl < slabs; ++sl) {
    const float* p = dxa + static_cast<int64_t>(sl) * n + i;
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w; v[4] += b.x; v[5] += b.y; v[6] += b.z;
    v[7] += b.w;
  }
  *reinterpret_cast<uint4*>(dx + i) = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                                 pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
}

// wst[h][c] = c < vb ? w[h][v0 + c] : 0 for c < vbp (padded copy of a block)
__global__ __launch_bounds__(256) void voc_stage_kernel(const uint16_t* __restrict__ w, int64_t V,
                                                        int64_t v0, int vb, int vbp, int H,
                                                        uint16_t* __restrict__ wst) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(H) * vbp) return;
  const int64_t h = i / vbp;
  const int c = static_cast<int>(i - h * vbp);
  wst[i] = c < vb ? w[h * V + v0 + c] : uint16_t{0};
}

// dw[h][v0 + c] = dwst[h][c] for c < vb
__global__ __launch_bounds__(256) void voc_unstage_kernel(const uint16_t* __restrict__ dwst,
                                                          int vbp, int vb, int H, int64_t V,
                                                          int64_t v0, uint16_t* __restrict__ dw) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(H) * vb) return;
  const int64_t h = i / vb;
  const int c = static_cast<int>(i - h * vb);
  dw[h * V + v0 + c] = dwst[h * vbp + c];
}

__global__ __launch_bounds__(256) void voc_zero_bf16_kernel(uint16_t* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

bool staged(int64_t V) { return (V % 8) != 0; }

// K ranges of the dX product: enough (row tile x column tile x range) work
// items for about two per compute unit of a 256-CU device, each range at
// least 512 columns (a multiple of 64)
int64_t dx_kspan(int64_t N, int H, int64_t vblock) {
  const int64_t tiles = std::max<int64_t>(1, ceil_div(N, 256) * ceil_div(H, 256));
  int64_t S = std::min<int64_t>(8, std::max<int64_t>(1, ceil_div(512, tiles)));
  S = std::max<int64_t>(1, std::min<int64_t>(S, vblock / 512));
  return align_up(static_cast<size_t>(ceil_div(vblock, S)), 64);
}

}  // namespace

size_t vocab_fwd_ws_bytes(int64_t N, int H, int64_t V, int64_t vblock) {
  const int64_t vb = std::min(vblock, V);
  size_t b = align_up(sizeof(float) * 2 * static_cast<size_t>(N) * ceil_div(vb, 64), 256);  // pairs
  b += 3 * align_up(sizeof(float) * static_cast<size_t>(N), 256);  // running max, sum; target logit
  if (staged(V)) b += align_up(sizeof(uint16_t) * static_cast<size_t>(H) * align_up(vb, 8), 256);
  return b + 256;
}

size_t vocab_bwd_ws_bytes(int64_t N, int H, int64_t V, int64_t vblock) {
  const int64_t vb = std::min(vblock, V);
  const int64_t vbp = align_up(vb, 8);
  const int64_t slabs = ceil_div(vb, dx_kspan(N, H, vblock));
  size_t b = align_up(sizeof(uint16_t) * static_cast<size_t>(N) * vbp, 256);            // G
  b += align_up(sizeof(float) * static_cast<size_t>(slabs) * N * H, 256);                // dX slabs
  if (staged(V)) b += 2 * align_up(sizeof(uint16_t) * static_cast<size_t>(H) * vbp, 256);  // W, dW
  return b + 256;
}

hipError_t launch_vocab_fwd(const uint16_t* x, const uint16_t* w, const int32_t* target,
                            int64_t N, int H, int64_t V, int64_t vblock, float* loss, float* lse,
                            void* ws, hipStream_t s) {
  if (N == 0) return hipSuccess;
  const int64_t vbmax = std::min(vblock, V);
  char* p = static_cast<char*>(ws);
  float* part = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * 2 * static_cast<size_t>(N) * ceil_div(vbmax, 64), 256);
  float* m = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N), 256);
  float* sm = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N), 256);
  float* yt = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N), 256);
  uint16_t* wst = staged(V) ? reinterpret_cast<uint16_t*>(p) : nullptr;
  const int n = static_cast<int>(N);
  for (int64_t b0 = 0; b0 < V; b0 += vblock) {
    const int vb = static_cast<int>(std::min<int64_t>(vblock, V - b0));
    const uint16_t* wb = w;
    int64_t ldw = V, bc0 = b0;
    if (wst != nullptr) {
      const int vbp = static_cast<int>(align_up(vb, 8));
      voc_stage_kernel<<<static_cast<unsigned>(ceil_div(static_cast<int64_t>(H) * vbp, 256)), 256,
                         0, s>>>(w, V, b0, vb, vbp, H, wst);
      if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
      wb = wst;
      ldw = vbp;
      bc0 = 0;
    }
    if (hipError_t e = launch_vocab_logits_mfma(x, wb, ldw, bc0, b0, n, H, vb, target, part, yt, s);
        e != hipSuccess)
      return e;
    prof_begin(K_VOC_LSE, s);
    voc_merge_kernel<<<static_cast<unsigned>(ceil_div(N, 4)), 256, 0, s>>>(
        reinterpret_cast<const float2*>(part), static_cast<int>(ceil_div(vb, 64)), N, m, sm,
        b0 == 0);
    prof_end(K_VOC_LSE, s);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  voc_finalize_kernel<<<static_cast<unsigned>(ceil_div(N, 256)), 256, 0, s>>>(m, sm, yt, N, loss,
                                                                              lse);
  return hipGetLastError();
}

hipError_t launch_vocab_bwd(const uint16_t* x, const uint16_t* w, const int32_t* target,
                            const float* lse, const float* dloss, int64_t N, int H, int64_t V,
                            int64_t vblock, uint16_t* dx, uint16_t* dw, void* ws, hipStream_t s) {
  if (N == 0) {  // no tokens: the weight gradient is exact zeros (dx is empty)
    const int64_t nw = static_cast<int64_t>(H) * V;
    voc_zero_bf16_kernel<<<static_cast<unsigned>(ceil_div(nw, 256)), 256, 0, s>>>(dw, nw);
    return hipGetLastError();
  }
  const int64_t vbmax = std::min(vblock, V);
  const int64_t vbpmax = align_up(vbmax, 8);
  const int kspan = static_cast<int>(dx_kspan(N, H, vblock));
  const int slabs = static_cast<int>(ceil_div(vbmax, kspan));  // the first block fills them all
  char* p = static_cast<char*>(ws);
  uint16_t* G = reinterpret_cast<uint16_t*>(p);
  p += align_up(sizeof(uint16_t) * static_cast<size_t>(N) * vbpmax, 256);
  float* dxa = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(slabs) * N * H, 256);
  uint16_t* wst = nullptr;
  uint16_t* dwst = nullptr;
  if (staged(V)) {
    wst = reinterpret_cast<uint16_t*>(p);
    p += align_up(sizeof(uint16_t) * static_cast<size_t>(H) * vbpmax, 256);
    dwst = reinterpret_cast<uint16_t*>(p);
  }
  const int n = static_cast<int>(N);
  for (int64_t b0 = 0; b0 < V; b0 += vblock) {
    const int vb = static_cast<int>(std::min<int64_t>(vblock, V - b0));
    const int64_t gp = align_up(vb, 8);
    const uint16_t* wb = w;
    int64_t ldw = V, bc0 = b0;
    uint16_t* dwb = dw;
    int64_t ldd = V, cc0 = b0;
    if (wst != nullptr) {
      voc_stage_kernel<<<static_cast<unsigned>(ceil_div(static_cast<int64_t>(H) * gp, 256)), 256,
                         0, s>>>(w, V, b0, vb, static_cast<int>(gp), H, wst);
      if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
      wb = wst;
      ldw = gp;
      bc0 = 0;
      dwb = dwst;
      ldd = gp;
      cc0 = 0;
    }
    if (hipError_t e = launch_vocab_grad_mfma(x, wb, ldw, bc0, b0, n, H, vb, target, lse, dloss, G,
                                              gp, s);
        e != hipSuccess)
      return e;
    if (hipError_t e = launch_vocab_dx_mfma(G, gp, wb, ldw, bc0, n, H, vb, kspan, b0 == 0, dxa, s);
        e != hipSuccess)
      return e;
    if (hipError_t e = launch_vocab_dw_mfma(x, G, gp, n, H, vb, dwb, ldd, cc0, s); e != hipSuccess)
      return e;
    if (dwst != nullptr) {
      voc_unstage_kernel<<<static_cast<unsigned>(ceil_div(static_cast<int64_t>(H) * vb, 256)), 256,
                           0, s>>>(dwst, static_cast<int>(gp), vb, H, V, b0, dw);
      if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    }
  }
  const int64_t nx = N * H;
  voc_dx_sum_kernel<<<static_cast<unsigned>(ceil_div(nx / 8, 256)), 256, 0, s>>>(dxa, slabs, nx, dx);
  return hipGetLastError();
}

}  // namespace moe
