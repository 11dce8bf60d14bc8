// Router of the MoE layer on gfx950: logits and top-k softmax gates.
//
// Logits follow one fixed fp32 order (a fused-multiply-add chain over the
// hidden index ascending from +0.0f, then one add of the bias) so that the
// expert choice is reproducible bit for bit.  That forbids a split of the
// hidden dimension and any matrix-core reduction, so the logits are a
// register-blocked SIMT fp32 kernel: each thread owns a TM x TN block of
// (token, expert) chains; x and W_r chunks are staged through LDS.
#include "common.h"

namespace moe {
namespace {

constexpr int KC = 16;  // hidden-index chunk staged per LDS round

template <int TM, int TN, int TX, int TY>
__global__ __launch_bounds__(256) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                           const float* __restrict__ w,
                                                           const float* __restrict__ bias,
                                                           int64_t T, int d, int E,
                                                           float* __restrict__ logits) {
  static_assert(TX * TY == 256, "256 threads");
  constexpr int BT = TM * TY;  // tokens per block
  constexpr int BE = TN * TX;  // experts per block
  __shared__ __align__(16) float xs[KC][BT];
  __shared__ __align__(16) float ws[KC][BE];

  const int tid = threadIdx.x;
  const int tx = tid % TX, ty = tid / TX;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * BT;
  const int e0 = blockIdx.y * BE;

  float acc[TM][TN];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TN; ++b) acc[a][b] = +0.0f;

  for (int j0 = 0; j0 < d; j0 += KC) {
    const int kc = min(KC, d - j0);
    // x chunk: BT tokens x KC hidden values, 4 bf16 (8 bytes) per load
    for (int q = tid; q < BT * KC / 4; q += 256) {
      const int tt = q / (KC / 4);
      const int jq = (q % (KC / 4)) * 4;
      const int64_t t = t0 + tt;
      uint2 v = make_uint2(0u, 0u);
      if (t < T && jq < kc) v = *reinterpret_cast<const uint2*>(x + t * d + j0 + jq);
      xs[jq + 0][tt] = bf16_lo(v.x);
      xs[jq + 1][tt] = bf16_hi(v.x);
      xs[jq + 2][tt] = bf16_lo(v.y);
      xs[jq + 3][tt] = bf16_hi(v.y);
    }
    // W_r chunk: KC rows x BE experts
    for (int q = tid; q < KC * BE; q += 256) {
      const int jj = q / BE, ee = q % BE;
      const int e = e0 + ee;
      ws[jj][ee] = (jj < kc && e < E) ? w[static_cast<int64_t>(j0 + jj) * E + e] : 0.0f;
    }
    __syncthreads();
    for (int jj = 0; jj < kc; ++jj) {
      float xv[TM], wv[TN];
#pragma unroll
      for (int a = 0; a < TM; ++a) xv[a] = xs[jj][ty * TM + a];
#pragma unroll
      for (int b = 0; b < TN; ++b) wv[b] = ws[jj][tx * TN + b];
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TN; ++b) acc[a][b] = __builtin_fmaf(xv[a], wv[b], acc[a][b]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    const int64_t t = t0 + ty * TM + a;
    if (t >= T) continue;
#pragma unroll
    for (int b = 0; b < TN; ++b) {
      const int e = e0 + tx * TN + b;
      if (e >= E) continue;
      float v = acc[a][b];
      if (bias) v = v + bias[e];
      logits[t * E + e] = v;
    }
  }
}

// One wave per token: k rounds of a wave-wide arg-max over the not yet
// chosen experts, ordered by (logit descending, index ascending).  Lane i
// keeps slot i.  Gates: softmax over all E (renorm = 0) or over the chosen k.
template <int NV>
__global__ __launch_bounds__(256) void route_topk_kernel(const float* __restrict__ logits,
                                                         int64_t T, int E, int k, int renorm,
                                                         int32_t* __restrict__ idx,
                                                         float* __restrict__ gate) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* l = logits + t * E;
  float v[NV];
  uint32_t taken = 0;
#pragma unroll
  for (int i = 0; i < NV; ++i) {
    const int e = lane + 64 * i;
    if (e < E) {
      v[i] = l[e];
    } else {
      v[i] = -__builtin_huge_valf();
      taken |= 1u << i;
    }
  }
  float my_v = 0.0f;
  int my_e = 0;
  for (int s = 0; s < k; ++s) {
    float bv = -__builtin_huge_valf();
    int be = 0x7fffffff;
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int e = lane + 64 * i;
      const bool free_ = !((taken >> i) & 1u);
      if (free_ && (v[i] > bv || (v[i] == bv && e < be))) {
        bv = v[i];
        be = e;
      }
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const float ov = __shfl_xor(bv, o, 64);
      const int oe = __shfl_xor(be, o, 64);
      if (ov > bv || (ov == bv && oe < be)) {
        bv = ov;
        be = oe;
      }
    }
    if ((be & 63) == lane) taken |= 1u << (be >> 6);
    if (lane == s) {
      my_v = bv;
      my_e = be;
    }
  }
  const float m = __shfl(my_v, 0, 64);
  float part = 0.0f;
  if (renorm == 0) {
#pragma unroll
    for (int i = 0; i < NV; ++i)
      if (lane + 64 * i < E) part += expf(v[i] - m);
  } else if (lane < k) {
    part = expf(my_v - m);
  }
  const float den = wave_sum(part);
  if (lane < k) {
    idx[t * k + lane] = my_e;
    gate[t * k + lane] = expf(my_v - m) / den;
  }
}

template <int TM, int TN, int TX, int TY>
hipError_t run_logits(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                      int E, float* logits, hipStream_t s) {
  constexpr int BT = TM * TY, BE = TN * TX;
  dim3 grid(static_cast<unsigned>(ceil_div(T, BT)), static_cast<unsigned>(ceil_div(E, BE)));
  prof_begin(K_ROUTE_LOGITS, s);
  route_logits_kernel<TM, TN, TX, TY><<<grid, 256, 0, s>>>(x, w, bias, T, d, E, logits);
  prof_end(K_ROUTE_LOGITS, s);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_route(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                        int E, int k, int renorm, int32_t* idx, float* gate, float* logits,
                        hipStream_t s) {
  if (T == 0) return hipSuccess;
  // Largest register block that still gives >= 2 blocks per CU.
  const int64_t want = 512;
  hipError_t err;
  auto nblk = [&](int bt, int be) { return ceil_div(T, bt) * ceil_div(E, be); };
  if (nblk(64, 128) >= want && E > 64)
    err = run_logits<8, 4, 32, 8>(x, w, bias, T, d, E, logits, s);
  else if (nblk(64, 64) >= want)
    err = run_logits<4, 4, 16, 16>(x, w, bias, T, d, E, logits, s);
  else
    err = run_logits<2, 2, 16, 16>(x, w, bias, T, d, E, logits, s);
  if (err != hipSuccess) return err;

  const unsigned grid = static_cast<unsigned>(ceil_div(T, 4));
  prof_begin(K_ROUTE_TOPK, s);
  if (E <= 64)
    route_topk_kernel<1><<<grid, 256, 0, s>>>(logits, T, E, k, renorm, idx, gate);
  else if (E <= 128)
    route_topk_kernel<2><<<grid, 256, 0, s>>>(logits, T, E, k, renorm, idx, gate);
  else if (E <= 256)
    route_topk_kernel<4><<<grid, 256, 0, s>>>(logits, T, E, k, renorm, idx, gate);
  else if (E <= 512)
    route_topk_kernel<8><<<grid, 256, 0, s>>>(logits, T, E, k, renorm, idx, gate);
  else
    route_topk_kernel<16><<<grid, 256, 0, s>>>(logits, T, E, k, renorm, idx, gate);
  prof_end(K_ROUTE_TOPK, s);
  return hipGetLastError();
}

}  // namespace moe
