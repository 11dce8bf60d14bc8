// Router of the MoE layer on gfx950: logits and top-k softmax gates.
//
// Logits follow one fixed fp32 order (a fused-multiply-add chain over the
// hidden index ascending from +0.0f, then one add of the bias) so that the
// expert choice is reproducible bit for bit.  That forbids a split of the
// hidden dimension and any matrix-core reduction, so the logits are a
// register-blocked SIMT fp32 kernel: each lane owns TM x TE (token, expert)
// chains; x and W_r chunks are staged through LDS.
#include "common.h"

namespace moe {
namespace {

constexpr int KC = 32;  // hidden-index chunk staged per LDS round

// Lane = expert (experts lane + 64 i, i < TE), TM tokens per wave, 4 waves
// per block (BT = 4 TM tokens).  Per hidden index j a lane reads its TE
// router weights (LDS, distinct per lane) and the wave's TM token values
// (LDS broadcast, fp32), then advances TM x TE independent fma chains.
template <int TM, int TE>
__global__ __launch_bounds__(256) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                           const float* __restrict__ w,
                                                           const float* __restrict__ bias,
                                                           int64_t T, int d, int E,
                                                           float* __restrict__ logits) {
  constexpr int BT = 4 * TM;
  __shared__ __align__(16) float xs[KC][BT];
  __shared__ __align__(16) float ws[KC][64 * TE];
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * BT;
  float acc[TM][TE];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TE; ++b) acc[a][b] = +0.0f;

  for (int j0 = 0; j0 < d; j0 += KC) {
    const int kc = min(KC, d - j0);  // a multiple of 8
    // x chunk -> fp32, transposed to [j][token]: 8 bf16 (16 bytes) per load
    for (int q = tid; q < BT * (KC / 8); q += 256) {
      const int tt = q / (KC / 8), jq = (q % (KC / 8)) * 8;
      const int64_t t = t0 + tt;
      uint4 v = make_uint4(0u, 0u, 0u, 0u);
      if (t < T && jq < kc) v = *reinterpret_cast<const uint4*>(x + t * d + j0 + jq);
      xs[jq + 0][tt] = bf16_lo(v.x); xs[jq + 1][tt] = bf16_hi(v.x);
      xs[jq + 2][tt] = bf16_lo(v.y); xs[jq + 3][tt] = bf16_hi(v.y);
      xs[jq + 4][tt] = bf16_lo(v.z); xs[jq + 5][tt] = bf16_hi(v.z);
      xs[jq + 6][tt] = bf16_lo(v.w); xs[jq + 7][tt] = bf16_hi(v.w);
    }
    // W_r chunk: KC rows x (64 TE) experts, coalesced along experts
    for (int q = tid; q < KC * 64 * TE; q += 256) {
      const int jj = q / (64 * TE), ee = q % (64 * TE);
      ws[jj][ee] = (jj < kc && ee < E) ? w[static_cast<int64_t>(j0 + jj) * E + ee] : 0.0f;
    }
    __syncthreads();
    auto step = [&](int jj) {
      float xv[TM], wr[TE];
#pragma unroll
      for (int a = 0; a < TM; ++a) xv[a] = xs[jj][wv * TM + a];  // broadcast
#pragma unroll
      for (int b = 0; b < TE; ++b) wr[b] = ws[jj][lane + 64 * b];
#pragma unroll
      for (int a = 0; a < TM; ++a)
#pragma unroll
        for (int b = 0; b < TE; ++b) acc[a][b] = __builtin_fmaf(xv[a], wr[b], acc[a][b]);
    };
    if (kc == KC) {
#pragma unroll
      for (int jj = 0; jj < KC; ++jj) step(jj);
    } else {
      for (int j8 = 0; j8 < kc; j8 += 8) {
#pragma unroll
        for (int u = 0; u < 8; ++u) step(j8 + u);
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    const int64_t t = t0 + wv * TM + a;
    if (t >= T) continue;
#pragma unroll
    for (int b = 0; b < TE; ++b) {
      const int e = lane + 64 * b;
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

template <int TM, int TE>
hipError_t run_logits(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                      int E, float* logits, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(ceil_div(T, 4 * TM));
  prof_begin(K_ROUTE_LOGITS, s);
  route_logits_kernel<TM, TE><<<grid, 256, 0, s>>>(x, w, bias, T, d, E, logits);
  prof_end(K_ROUTE_LOGITS, s);
  return hipGetLastError();
}

// Tokens per wave: the largest of 8, 4, 2 that still gives every CU a
// workgroup.
template <int TE>
hipError_t pick_logits(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                       int E, float* logits, hipStream_t s) {
  if (ceil_div(T, 32) >= 256) return run_logits<8, TE>(x, w, bias, T, d, E, logits, s);
  if (ceil_div(T, 16) >= 256) return run_logits<4, TE>(x, w, bias, T, d, E, logits, s);
  return run_logits<2, TE>(x, w, bias, T, d, E, logits, s);
}

}  // namespace

hipError_t launch_route(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                        int E, int k, int renorm, int32_t* idx, float* gate, float* logits,
                        hipStream_t s) {
  if (T == 0) return hipSuccess;
  hipError_t err;
  if (E <= 64) err = pick_logits<1>(x, w, bias, T, d, E, logits, s);
  else if (E <= 128) err = pick_logits<2>(x, w, bias, T, d, E, logits, s);
  else if (E <= 256) err = pick_logits<4>(x, w, bias, T, d, E, logits, s);
  else if (E <= 512) err = pick_logits<8>(x, w, bias, T, d, E, logits, s);
  else err = pick_logits<16>(x, w, bias, T, d, E, logits, s);
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
