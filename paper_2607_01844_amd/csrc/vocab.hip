// Blockwise vocabulary projection loss (the MoP paper's data-tensor-parallel
// projection, Sec. 3.4 eq. voc-fwd-loss, on one device: P = 1, blocks of the
// vocabulary instead of ranks).  Y = X W_voc is never materialised: the
// forward walks the vocabulary in blocks of `vblock` columns, each block's
// logits (fp32) feed a running max / sum of exponentials per token (an
// online log-sum-exp, blocks merged in order, so the result is bitwise
// reproducible); the backward recomputes each block's logits and turns them
// into that block's logit gradients, from which it accumulates dX (fp32) and
// writes the block's columns of dW.
//
// The three products per block are plain dense GEMMs and go to rocBLAS (bf16
// operands, fp32 accumulation); everything between them is the kernels here.
#include "blas.h"

namespace moe {
namespace {

constexpr int VT = 256;  // threads per block of the row kernels (one token row per block)
constexpr int VU = 4;    // float4 loads in flight per thread

// Merge of two (max, sum of exp(y - max)) pairs; an empty pair is (-inf, 0).
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  const float mm = fmaxf(m, m2);
  if (mm == -__builtin_huge_valf()) return;  // both empty
  s = s * expf(m - mm) + s2 * expf(m2 - mm);
  m = mm;
}

// One block per token row n of a block of logits Y [N][pitch] (columns
// [0, vb) valid, pitch a multiple of 4 so rows are 16-byte aligned): a single
// pass keeps a running (max, sum) per thread over float4 groups, the block
// combines the threads' pairs in a fixed tree, and thread 0 merges the
// block's pair into the row's running (m, s) (blocks in order: bitwise
// reproducible).  The target's logit is taken from the block that holds it.
__global__ __launch_bounds__(VT) void voc_block_lse_kernel(const float* __restrict__ Y, int vb,
                                                           int pitch, int64_t b0,
                                                           const int32_t* __restrict__ target,
                                                           float* __restrict__ m,
                                                           float* __restrict__ s,
                                                           float* __restrict__ yt, int first) {
  __shared__ float sm[VT / 64], ss[VT / 64];
  const int64_t n = blockIdx.x;
  const float4* row = reinterpret_cast<const float4*>(Y + n * pitch);
  const int nq = (vb + 3) >> 2;
  constexpr float NEG = -__builtin_huge_valf();
  float tm = NEG, ts = 0.0f;
  for (int q0 = threadIdx.x; q0 < nq; q0 += VT * VU) {
    float4 v[VU];
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int q = q0 + u * VT;
      v[u] = q < nq ? row[q] : make_float4(NEG, NEG, NEG, NEG);
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int c = (q0 + u * VT) * 4;  // columns c..c+3; those >= vb are padding
      const float a0 = v[u].x, a1 = c + 1 < vb ? v[u].y : NEG, a2 = c + 2 < vb ? v[u].z : NEG,
                  a3 = c + 3 < vb ? v[u].w : NEG;
      const float gm = fmaxf(fmaxf(a0, a1), fmaxf(a2, a3));
      if (gm == NEG) continue;
      if (gm > tm) {
        ts *= expf(tm - gm);
        tm = gm;
      }
      ts += (expf(a0 - tm) + expf(a1 - tm)) + (expf(a2 - tm) + expf(a3 - tm));
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float m2 = __shfl_xor(tm, o, 64), s2 = __shfl_xor(ts, o, 64);
    lse_merge(tm, ts, m2, s2);
  }
  const int wv = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sm[wv] = tm;
    ss[wv] = ts;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float bm = sm[0], bs = ss[0];
#pragma unroll
    for (int k = 1; k < VT / 64; ++k) lse_merge(bm, bs, sm[k], ss[k]);
    if (first) {
      m[n] = bm;
      s[n] = bs;
    } else {
      float rm = m[n], rs = s[n];
      lse_merge(rm, rs, bm, bs);
      m[n] = rm;
      s[n] = rs;
    }
    const int64_t t = target[n];
    if (t >= b0 && t < b0 + vb) yt[n] = Y[n * pitch + (t - b0)];
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

// One block per token row: G[n][v] = bf16( dloss_n * ([b0 + v == t_n] -
// exp(Y[n][v] - lse_n)) ), the gradient of loss_n with respect to this
// block's logits, four columns per thread and store; padding columns
// [vb, pitch) get zeros.
__global__ __launch_bounds__(VT) void voc_grad_kernel(const float* __restrict__ Y, int vb,
                                                      int pitch, int64_t b0,
                                                      const int32_t* __restrict__ target,
                                                      const float* __restrict__ lse,
                                                      const float* __restrict__ dloss,
                                                      uint16_t* __restrict__ G) {
  const int64_t n = blockIdx.x;
  const float4* row = reinterpret_cast<const float4*>(Y + n * pitch);
  uint2* grow = reinterpret_cast<uint2*>(G + n * pitch);
  const int nq = pitch >> 2;
  const float l = lse[n], dl = dloss[n];
  const int64_t tc = static_cast<int64_t>(target[n]) - b0;  // target column in this block
  for (int q0 = threadIdx.x; q0 < nq; q0 += VT * VU) {
    float4 v[VU];
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int q = q0 + u * VT;
      v[u] = q < nq ? row[q] : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int u = 0; u < VU; ++u) {
      const int q = q0 + u * VT;
      if (q >= nq) break;
      const int c = q * 4;
      float g[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
      for (int i = 0; i < 4; ++i)
        g[i] = c + i < vb ? dl * ((c + i == tc ? 1.0f : 0.0f) - expf(g[i] - l)) : 0.0f;
      grow[q] = make_uint2(pack_bf16x2(g[0], g[1]), pack_bf16x2(g[2], g[3]));
    }
  }
}

__global__ __launch_bounds__(256) void voc_fill_kernel(float* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = 0.0f;
}

__global__ __launch_bounds__(256) void voc_zero_bf16_kernel(uint16_t* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = 0;
}

__global__ __launch_bounds__(256) void voc_to_bf16_kernel(const float* __restrict__ a, int64_t n,
                                                          uint16_t* __restrict__ b) {
  const int64_t i = (static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x) * 2;
  if (i >= n) return;  // n is even (H is a multiple of 8)
  *reinterpret_cast<uint32_t*>(b + i) = pack_bf16x2(a[i], a[i + 1]);
}

}  // namespace

size_t vocab_fwd_ws_bytes(int64_t N, int64_t vblock) {
  return align_up(sizeof(float) * static_cast<size_t>(N) * vblock, 256) +
         3 * align_up(sizeof(float) * static_cast<size_t>(N), 256) + kBlasWs + 256;
}

size_t vocab_bwd_ws_bytes(int64_t N, int H, int64_t vblock) {
  return align_up(sizeof(float) * static_cast<size_t>(N) * vblock, 256) +
         align_up(sizeof(uint16_t) * static_cast<size_t>(N) * vblock, 256) +
         align_up(sizeof(float) * static_cast<size_t>(N) * H, 256) + kBlasWs + 256;
}

// Row-major [r][c] with pitch ld is column-major c x r with the same pitch,
// which is how every product below is handed to rocBLAS.  A block's logits
// and logit gradients use a row pitch of vb rounded up to 8 columns, so
// every row starts 16-byte aligned; the padding columns are never read by
// the products.
hipError_t launch_vocab_fwd(const uint16_t* x, const uint16_t* w, const int32_t* target,
                            int64_t N, int H, int64_t V, int64_t vblock, float* loss, float* lse,
                            void* ws, hipStream_t s) {
  if (N == 0) return hipSuccess;
  char* p = static_cast<char*>(ws);
  float* Y = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N) * vblock, 256);
  float* m = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N), 256);
  float* sm = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N), 256);
  float* yt = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N), 256);
  void* bws = p;
  BlasLease B(s, bws);
  if (hipError_t e = B.status(); e != hipSuccess) return e;
  const unsigned gr = static_cast<unsigned>(N);
  for (int64_t b0 = 0; b0 < V; b0 += vblock) {
    const int vb = static_cast<int>(std::min<int64_t>(vblock, V - b0));
    const int pitch = static_cast<int>(align_up(vb, 8));
    // Y[N][vb] = X[N][H] W[H][b0 : b0 + vb]
    if (hipError_t e = gemm_bf16(B.handle(), false, false, vb, static_cast<int>(N), H, w + b0,
                                 static_cast<int>(V), 0, x, H, 0, 0.0f, Y, false, pitch, 0);
        e != hipSuccess)
      return e;
    prof_begin(K_VOC_LSE, s);
    voc_block_lse_kernel<<<gr, VT, 0, s>>>(Y, vb, pitch, b0, target, m, sm, yt, b0 == 0);
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
  if (N == 0) {  // no tokens: both gradients are exact zeros
    const int64_t nw = static_cast<int64_t>(H) * V;
    voc_zero_bf16_kernel<<<static_cast<unsigned>(ceil_div(nw, 256)), 256, 0, s>>>(dw, nw);
    return hipGetLastError();
  }
  char* p = static_cast<char*>(ws);
  float* Y = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N) * vblock, 256);
  uint16_t* G = reinterpret_cast<uint16_t*>(p);
  p += align_up(sizeof(uint16_t) * static_cast<size_t>(N) * vblock, 256);
  float* dxa = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * static_cast<size_t>(N) * H, 256);
  void* bws = p;
  BlasLease B(s, bws);
  if (hipError_t e = B.status(); e != hipSuccess) return e;
  const int64_t nx = N * H;
  voc_fill_kernel<<<static_cast<unsigned>(ceil_div(nx, 256)), 256, 0, s>>>(dxa, nx);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  const int n = static_cast<int>(N), ldw = static_cast<int>(V);
  for (int64_t b0 = 0; b0 < V; b0 += vblock) {
    const int vb = static_cast<int>(std::min<int64_t>(vblock, V - b0));
    const int pitch = static_cast<int>(align_up(vb, 8));
    // Y[N][vb] = X W[:, b0 : b0 + vb]   (recomputed)
    if (hipError_t e = gemm_bf16(B.handle(), false, false, vb, n, H, w + b0, ldw, 0, x, H, 0, 0.0f,
                                 Y, false, pitch, 0);
        e != hipSuccess)
      return e;
    prof_begin(K_VOC_GRAD, s);
    voc_grad_kernel<<<static_cast<unsigned>(N), VT, 0, s>>>(Y, vb, pitch, b0, target, lse, dloss,
                                                           G);
    prof_end(K_VOC_GRAD, s);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
    // dX[N][H] += G[N][vb] W[:, b0 : b0 + vb]^T
    if (hipError_t e = gemm_bf16(B.handle(), true, false, H, n, vb, w + b0, ldw, 0, G, pitch, 0,
                                 1.0f, dxa, false, H, 0);
        e != hipSuccess)
      return e;
    // dW[:, b0 : b0 + vb] = X^T G
    if (hipError_t e = gemm_bf16(B.handle(), false, true, vb, H, n, G, pitch, 0, x, H, 0, 0.0f,
                                 dw + b0, true, ldw, 0);
        e != hipSuccess)
      return e;
  }
  voc_to_bf16_kernel<<<static_cast<unsigned>(ceil_div(nx / 2, 256)), 256, 0, s>>>(dxa, nx, dx);
  return hipGetLastError();
}

}  // namespace moe
