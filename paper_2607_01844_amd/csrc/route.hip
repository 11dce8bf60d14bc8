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

// Lane = expert (experts lane + 64 b, b < TE); a wave owns TM tokens, a block
// four waves.  The TM token values are uniform across the wave, so they come
// in through scalar loads (8 bf16 per load) and feed the FMAs as scalar
// operands; each lane reads only its own TE router weights from LDS.  W_r
// is staged in chunks of KC hidden indices, double-buffered: the next chunk
// is fetched into registers while the current one is consumed.
template <int TM, int TE, int KC>
__global__ __launch_bounds__(256) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                           const float* __restrict__ w,
                                                           const float* __restrict__ bias,
                                                           int64_t T, int d, int E,
                                                           float* __restrict__ logits) {
  constexpr int EW = 64 * TE;            // experts covered by one block row
  constexpr int NW = KC * EW / 256;      // W_r values each thread stages per chunk
  static_assert(KC % 8 == 0 && (KC * EW) % 256 == 0, "chunk shape");
  __shared__ __align__(16) float ws[2][KC][EW];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t tw = static_cast<int64_t>(blockIdx.x) * (4 * TM) + wv * TM;
  const uint4* xr[TM];
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    const int64_t t = tw + a < T ? tw + a : T - 1;  // tail rows recompute row T-1
    xr[a] = reinterpret_cast<const uint4*>(x + t * d);
  }
  float acc[TM][TE];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TE; ++b) acc[a][b] = +0.0f;

  float wr[NW];
  auto fetch = [&](int j0) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int q = tid + 256 * i, jj = q / EW, ee = q % EW;
      wr[i] = (j0 + jj < d && ee < E) ? w[static_cast<int64_t>(j0 + jj) * E + ee] : 0.0f;
    }
  };
  auto stash = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      const int q = tid + 256 * i;
      ws[buf][q / EW][q % EW] = wr[i];
    }
  };
  const int nch = (d + KC - 1) / KC;
  fetch(0);
  stash(0);
  __syncthreads();
  for (int c = 0; c < nch; ++c) {
    const int j0 = c * KC, kc = min(KC, d - j0);  // kc is a multiple of 8
    if (c + 1 < nch) fetch(j0 + KC);
    const int buf = c & 1;
    for (int g = 0; g < kc; g += 8) {
      uint4 xv[TM];
#pragma unroll
      for (int a = 0; a < TM; ++a) xv[a] = xr[a][(j0 + g) >> 3];  // uniform: scalar load
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float wl[TE];
#pragma unroll
        for (int b = 0; b < TE; ++b) wl[b] = ws[buf][g + u][lane + 64 * b];
#pragma unroll
        for (int a = 0; a < TM; ++a) {
          const uint32_t pr = u < 2 ? xv[a].x : u < 4 ? xv[a].y : u < 6 ? xv[a].z : xv[a].w;
          const float xa = (u & 1) ? bf16_hi(pr) : bf16_lo(pr);
#pragma unroll
          for (int b = 0; b < TE; ++b) acc[a][b] = __builtin_fmaf(xa, wl[b], acc[a][b]);
        }
      }
    }
    if (c + 1 < nch) stash(buf ^ 1);
    __syncthreads();
  }
#pragma unroll
  for (int a = 0; a < TM; ++a) {
    const int64_t t = tw + a;
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
  constexpr int KC = (64 / TE) >= 8 ? (64 / TE) / 8 * 8 : 8;
  const unsigned grid = static_cast<unsigned>(ceil_div(T, 4 * TM));
  prof_begin(K_ROUTE_LOGITS, s);
  route_logits_kernel<TM, TE, KC><<<grid, 256, 0, s>>>(x, w, bias, T, d, E, logits);
  prof_end(K_ROUTE_LOGITS, s);
  return hipGetLastError();
}

// Tokens per wave: the largest of 8, 4, 2, 1 that keeps TM * TE <= 32
// chains per lane and still launches about 2048 waves (two per SIMD), so
// that one wave's scalar-load latency is covered by the other's FMAs.
template <int TE>
hipError_t pick_logits(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                       int E, float* logits, hipStream_t s) {
  if constexpr (TE <= 4)
    if (T >= 8 * 2048) return run_logits<8, TE>(x, w, bias, T, d, E, logits, s);
  if constexpr (TE <= 8)
    if (T >= 4 * 2048) return run_logits<4, TE>(x, w, bias, T, d, E, logits, s);
  if (T >= 2 * 2048) return run_logits<2, TE>(x, w, bias, T, d, E, logits, s);
  return run_logits<1, TE>(x, w, bias, T, d, E, logits, s);
}

}  // namespace

hipError_t launch_route(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                        int E, int k, int renorm, int32_t* idx, float* gate, float* logits,
                        hipStream_t s) {
  if (T == 0) return hipSuccess;
  hipError_t err;
  switch ((E + 63) / 64) {
    case 1: err = pick_logits<1>(x, w, bias, T, d, E, logits, s); break;
    case 2: err = pick_logits<2>(x, w, bias, T, d, E, logits, s); break;
    case 3: err = pick_logits<3>(x, w, bias, T, d, E, logits, s); break;
    case 4: err = pick_logits<4>(x, w, bias, T, d, E, logits, s); break;
    case 5: case 6: err = pick_logits<6>(x, w, bias, T, d, E, logits, s); break;
    case 7: case 8: err = pick_logits<8>(x, w, bias, T, d, E, logits, s); break;
    case 9: case 10: case 11: case 12: err = pick_logits<12>(x, w, bias, T, d, E, logits, s); break;
    default: err = pick_logits<16>(x, w, bias, T, d, E, logits, s); break;
  }
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
