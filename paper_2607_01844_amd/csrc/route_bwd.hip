// Router backward on gfx950.  The router is a dense weight (W_r, optional
// bias) feeding the top-k softmax gates, so its gradient is the chain
//   gate gradients -> logit gradients (softmax Jacobian at the chosen slots)
//   -> dW_r = x^T dlogits, dbias = column sums of dlogits,
//      dx_router = dlogits W_r^T  (added to the expert path's dx).
// Fixed summation orders throughout, so results are bitwise reproducible.
// The two contractions (2 T d E FLOP each) run on the fp32 vector ALUs when
// they are small.  Large ones (a trillion-scale share: T = 16384, d = 7168,
// E = 384) go to the bf16 matrix cores without losing fp32 precision: every
// fp32 operand v is split into bf16 hi = bf16(v) and lo = bf16(v - hi)
// (|v - hi - lo| <= 2^-17 |v|), and the products are taken as
//   dW_r = x^T (hi + lo)        (x is exactly bf16),
//   dx_router = hi_d hi_w + hi_d lo_w + lo_d hi_w
// with fp32 accumulation, on the library's grouped GEMM kernel (dense
// modes); the token range of dW_r is cut into chunks whose partial sums are
// added in chunk order.
#include <algorithm>

#include "common.h"

namespace moe {
namespace {

// One wave per token; lane holds experts lane + 64 i.
//   renorm = 0 (gates = softmax over all E at the chosen experts):
//     dl_e = -p_e s + sum_{i: e_i = e} dgate_i gate_i,  s = sum_i dgate_i gate_i
//   renorm = 1 (gates = softmax over the k chosen logits):
//     dl_{e_i} = gate_i (dgate_i - s), 0 for experts not chosen.
// p_e is recomputed from the logits the forward pass saved, as the forward
// computed it (max-shifted exponentials over all E).
template <int NV>
__global__ __launch_bounds__(256) void route_dlogits_kernel(const float* __restrict__ logits,
                                                            const int32_t* __restrict__ idx,
                                                            const float* __restrict__ gate,
                                                            const float* __restrict__ dgate,
                                                            int64_t T, int E, int k, int renorm,
                                                            float* __restrict__ dl) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const float* l = logits + t * E;
  const int32_t* it = idx + t * k;
  const float* gt = gate + t * k;
  const float* dg = dgate + t * k;
  float s = 0.0f;
  for (int i = 0; i < k; ++i) s = __builtin_fmaf(dg[i], gt[i], s);
  float v[NV];
  if (renorm == 0) {
    float m = -__builtin_huge_valf();
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int e = lane + 64 * j;
      v[j] = e < E ? l[e] : -__builtin_huge_valf();
      m = fmaxf(m, v[j]);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
    float part = 0.0f;
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if (lane + 64 * j < E) part += expf(v[j] - m);
    const float den = wave_sum(part);
#pragma unroll
    for (int j = 0; j < NV; ++j) v[j] = -(expf(v[j] - m) / den) * s;
  } else {
#pragma unroll
    for (int j = 0; j < NV; ++j) v[j] = 0.0f;
  }
  for (int i = 0; i < k; ++i) {
    const int e = it[i];
    if ((e & 63) != lane) continue;
    const float g = gt[i], d = dg[i];
#pragma unroll
    for (int j = 0; j < NV; ++j)
      if ((e >> 6) == j) v[j] = renorm == 0 ? v[j] + d * g : g * (d - s);
  }
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    const int e = lane + 64 * j;
    if (e < E) dl[t * E + e] = v[j];
  }
}

// dW_r partials: part[c][j][e] = sum over tokens t of chunk c (ascending) of
// float(x[t][j]) * dl[t][e].  Block = 64 hidden rows x 64 experts, thread =
// 4 x 4 outputs; x and dl are staged 32 tokens at a time through LDS.  With
// one chunk the block writes dw_r directly.  Blocks of hidden-row tile 0
// also produce the bias partials (sum over the chunk of dl[t][e]).
constexpr int RB_J = 64, RB_E = 64, RB_T = 32;
__global__ __launch_bounds__(256) void route_dw_kernel(const uint16_t* __restrict__ x,
                                                       const float* __restrict__ dl, int64_t T,
                                                       int d, int E, int64_t chunk,
                                                       float* __restrict__ part,
                                                       float* __restrict__ bpart) {
  __shared__ __align__(16) float xs[RB_T][RB_J];
  __shared__ __align__(16) float ds[RB_T][RB_E];
  const int tid = threadIdx.x;
  const int j0 = blockIdx.x * RB_J, e0 = blockIdx.y * RB_E, c = blockIdx.z;
  const int64_t tb = c * chunk, te = min(T, tb + chunk);
  const int tj = tid >> 4, tq = tid & 15;  // outputs j0 + 4 tj + 0..3, e0 + 4 tq + 0..3
  float acc[4][4] = {};
  float bacc[4] = {};
  const bool do_bias = bpart != nullptr && blockIdx.x == 0 && tj == 0;
  // staging: x row r = tid / 8 of the 32, columns 8 (tid % 8) .. +7 (one 16-byte load);
  // dl row r, columns 4 (tid % 16) .. +3 and rows r and r + 16
  const int xr = tid >> 3, xc = (tid & 7) * 8;
  const int dr = tid >> 4, dc = (tid & 15) * 4;
  for (int64_t t0 = tb; t0 < te; t0 += RB_T) {
    {
      const int64_t t = t0 + xr;
      uint4 u = make_uint4(0u, 0u, 0u, 0u);
      if (t < te && j0 + xc < d) u = *reinterpret_cast<const uint4*>(x + t * d + j0 + xc);
      float4* o = reinterpret_cast<float4*>(&xs[xr][xc]);
      o[0] = make_float4(bf16_lo(u.x), bf16_hi(u.x), bf16_lo(u.y), bf16_hi(u.y));
      o[1] = make_float4(bf16_lo(u.z), bf16_hi(u.z), bf16_lo(u.w), bf16_hi(u.w));
    }
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = dr + 16 * h;
      const int64_t t = t0 + r;
      float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
      if (t < te) {
        const float* p = dl + t * E + e0 + dc;
        const int n = E - (e0 + dc);
        if (n >= 4 && (E & 3) == 0) {
          v = *reinterpret_cast<const float4*>(p);
        } else {
          if (n > 0) v.x = p[0];
          if (n > 1) v.y = p[1];
          if (n > 2) v.z = p[2];
          if (n > 3) v.w = p[3];
        }
      }
      *reinterpret_cast<float4*>(&ds[r][dc]) = v;
    }
    __syncthreads();
    const int nt = static_cast<int>(min<int64_t>(RB_T, te - t0));
    for (int r = 0; r < nt; ++r) {
      const float4 a = *reinterpret_cast<const float4*>(&xs[r][4 * tj]);
      const float4 b = *reinterpret_cast<const float4*>(&ds[r][4 * tq]);
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[p][q] = __builtin_fmaf(av[p], bv[q], acc[p][q]);
      if (do_bias) {
#pragma unroll
        for (int q = 0; q < 4; ++q) bacc[q] += bv[q];
      }
    }
    __syncthreads();
  }
  float* out = part + static_cast<int64_t>(c) * d * E;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int j = j0 + 4 * tj + p;
    if (j >= d) continue;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = e0 + 4 * tq + q;
      if (e < E) out[static_cast<int64_t>(j) * E + e] = acc[p][q];
    }
  }
  if (do_bias) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int e = e0 + 4 * tq + q;
      if (e < E) bpart[static_cast<int64_t>(c) * E + e] = bacc[q];
    }
  }
}

// dw[i] = sum over chunks c ascending of part[c][i] (n = d E values; the bias
// partials ride along as n_b more values).
__global__ __launch_bounds__(256) void route_dw_reduce_kernel(const float* __restrict__ part,
                                                              int64_t n, int chunks,
                                                              float* __restrict__ dw,
                                                              const float* __restrict__ bpart,
                                                              int nb, float* __restrict__ dbias) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) {
    float s = part[i];
    for (int c = 1; c < chunks; ++c) s += part[static_cast<int64_t>(c) * n + i];
    dw[i] = s;
  } else if (dbias != nullptr && i < n + nb) {
    const int64_t e = i - n;
    float s = bpart[e];
    for (int c = 1; c < chunks; ++c) s += bpart[static_cast<int64_t>(c) * nb + e];
    dbias[e] = s;
  }
}

// hi / lo bf16 parts of fp32 values: hi = bf16(v), lo = bf16(v - hi).
__device__ __forceinline__ void split_bf16(float v, uint16_t& hi, uint16_t& lo) {
  hi = static_cast<uint16_t>(f32_to_bf16_bits(v));
  lo = static_cast<uint16_t>(f32_to_bf16_bits(v - bf16_to_f32(hi)));
}
// dl [T][E] -> dl3 [T][ld3] = [hi | hi | lo] (E columns each), zeros in
// [3E, ld3): one product over the 3E columns against [hi; lo; hi] of W_r^T
// sums the three cross terms, and the dW_r product reads the first hi group
// and the lo group.
__global__ __launch_bounds__(256) void route_split_dl_kernel(const float* __restrict__ dl,
                                                             int64_t T, int E, int ld3,
                                                             uint16_t* __restrict__ dl3) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= T * ld3) return;
  const int64_t t = i / ld3;
  const int c = static_cast<int>(i - t * ld3);
  uint16_t out = 0;
  if (c < 3 * E) {
    const int grp = c / E, e = c - grp * E;
    uint16_t hi, lo;
    split_bf16(dl[t * E + e], hi, lo);
    out = grp == 2 ? lo : hi;
  }
  dl3[i] = out;
}
// W_r [d][E] -> w3 [3E][d] = [hi; lo; hi] of W_r^T
__global__ __launch_bounds__(256) void route_split_w_kernel(const float* __restrict__ w, int d,
                                                            int E, uint16_t* __restrict__ w3) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i >= static_cast<int64_t>(3) * E * d) return;
  const int64_t r = i / d;
  const int j = static_cast<int>(i - r * d);
  const int grp = static_cast<int>(r / E), e = static_cast<int>(r - static_cast<int64_t>(grp) * E);
  uint16_t hi, lo;
  split_bf16(w[static_cast<int64_t>(j) * E + e], hi, lo);
  w3[i] = grp == 1 ? lo : hi;
}
// bpart[c][e] = sum over the tokens of chunk c of dl[t][e].  Lane = expert
// (64 per block); wave w of the block's 16 sums the chunk's tokens t0 + w,
// t0 + w + 16, ... in ascending order, eight loads in flight, and the 16
// wave sums are then added in wave order (a fixed order: the result repeats
// bit for bit).
constexpr int DB_WAVES = 16;
__global__ __launch_bounds__(64 * DB_WAVES) void route_dbias_part_kernel(const float* __restrict__ dl,
                                                                         int64_t T, int E, int64_t chunk,
                                                                         float* __restrict__ bpart) {
  __shared__ float red[DB_WAVES][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int e = blockIdx.x * 64 + lane;
  const int c = blockIdx.y;
  const int64_t t0 = c * chunk, t1 = std::min(T, t0 + chunk);
  float acc = 0.0f;
  if (e < E) {
    int64_t t = t0 + wv;
    for (; t + 7 * DB_WAVES < t1; t += 8 * DB_WAVES) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = dl[(t + u * DB_WAVES) * E + e];
#pragma unroll
      for (int u = 0; u < 8; ++u) acc += v[u];
    }
    for (; t < t1; t += DB_WAVES) acc += dl[t * E + e];
  }
  red[wv][lane] = acc;
  __syncthreads();
  if (wv == 0 && e < E) {
    float sum = red[0][lane];
    for (int q = 1; q < DB_WAVES; ++q) sum += red[q][lane];
    bpart[static_cast<int64_t>(c) * E + e] = sum;
  }
}

// dx[t][j] = bf16( [float(dx[t][j]) +] sum over e ascending of dl[t][e] * W_r[j][e] ).
// Block = 64 tokens x 64 hidden columns, thread = 4 tokens x 4 columns; dl
// and W_r are staged transposed (expert-major) 32 experts at a time.
constexpr int RX_T = 64, RX_J = 64, RX_E = 32;
__global__ __launch_bounds__(256) void route_dx_kernel(const float* __restrict__ dl,
                                                       const float* __restrict__ w, int64_t T,
                                                       int d, int E, int accumulate,
                                                       uint16_t* __restrict__ dx) {
  __shared__ __align__(16) float dlT[RX_E][RX_T + 4];
  __shared__ __align__(16) float wT[RX_E][RX_J + 4];
  const int tid = threadIdx.x;
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * RX_T;
  const int j0 = blockIdx.y * RX_J;
  const int tt = tid >> 4, tq = tid & 15;  // tokens t0 + 4 tt + 0..3, columns j0 + 4 tq + 0..3
  float acc[4][4] = {};
  for (int e0 = 0; e0 < E; e0 += RX_E) {
    // 64 rows x 32 experts of each operand: thread loads rows r = tid / 4 (+0),
    // experts 8 (tid % 4) .. +7
    const int r = tid >> 2, c8 = (tid & 3) * 8;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int e = e0 + c8 + u;
      const int64_t t = t0 + r;
      const int j = j0 + r;
      dlT[c8 + u][r] = (t < T && e < E) ? dl[t * E + e] : 0.0f;
      wT[c8 + u][r] = (j < d && e < E) ? w[static_cast<int64_t>(j) * E + e] : 0.0f;
    }
    __syncthreads();
    const int ne = min(RX_E, E - e0);
    for (int q = 0; q < ne; ++q) {
      const float4 a = *reinterpret_cast<const float4*>(&dlT[q][4 * tt]);
      const float4 b = *reinterpret_cast<const float4*>(&wT[q][4 * tq]);
      const float av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
      for (int p = 0; p < 4; ++p)
#pragma unroll
        for (int s = 0; s < 4; ++s) acc[p][s] = __builtin_fmaf(av[p], bv[s], acc[p][s]);
    }
    __syncthreads();
  }
  const int j = j0 + 4 * tq;
  if (j >= d) return;  // d is a multiple of 8, so j .. j + 3 are all in range
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const int64_t t = t0 + 4 * tt + p;
    if (t >= T) continue;
    uint2* o = reinterpret_cast<uint2*>(dx + t * d + j);
    float v[4] = {acc[p][0], acc[p][1], acc[p][2], acc[p][3]};
    if (accumulate) {
      const uint2 u = *o;
      v[0] = bf16_lo(u.x) + v[0];
      v[1] = bf16_hi(u.x) + v[1];
      v[2] = bf16_lo(u.y) + v[2];
      v[3] = bf16_hi(u.y) + v[3];
    }
    *o = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
  }
}

__global__ __launch_bounds__(256) void route_zero_kernel(float* __restrict__ p, int64_t n) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (i < n) p[i] = 0.0f;
}

}  // namespace

// Token chunks of the dW_r reduction: enough blocks to fill the chip
// (about 2048), each chunk at least 256 tokens.
int route_bwd_chunks(int64_t T, int d, int E) {
  if (T <= 0) return 0;
  const int64_t tiles = ceil_div(d, RB_J) * ceil_div(E, RB_E);
  const int64_t want = ceil_div(2048, tiles);
  const int64_t most = ceil_div(T, 256);
  return static_cast<int>(std::max<int64_t>(1, std::min(want, most)));
}

namespace {
// the matrix-core path takes contractions of at least 2^28 multiply-adds
bool route_bwd_mfma(int64_t T, int d, int E) {
  return T * static_cast<int64_t>(d) * E >= (int64_t{1} << 28);
}
// matrix-core path: token chunks of dW_r (multiples of 64 tokens, at least
// 512), so that the chunks' products have about 512 output tiles of 256 x
// 256 between them
int64_t route_bwd_mfma_chunk(int64_t T, int d, int E) {
  const int64_t tiles = ceil_div(d, 256) * ceil_div(E, 128);
  const int64_t S = std::max<int64_t>(1, std::min(ceil_div(512, tiles), ceil_div(T, 512)));
  return static_cast<int64_t>(align_up(static_cast<size_t>(ceil_div(T, S)), 64));
}
int route_bwd_ld3(int E) { return static_cast<int>(align_up(static_cast<size_t>(3 * E), 8)); }
}  // namespace

size_t route_bwd_ws_bytes(int64_t T, int d, int E) {
  const bool mf = route_bwd_mfma(T, d, E);
  const int S = mf ? static_cast<int>(ceil_div(T, route_bwd_mfma_chunk(T, d, E)))
                   : route_bwd_chunks(T, d, E);
  size_t b = align_up(sizeof(float) * static_cast<size_t>(T) * E, 256);  // dlogits
  if (S > 1) {
    b += align_up(sizeof(float) * static_cast<size_t>(S) * d * E, 256);  // dW_r partials
    b += align_up(sizeof(float) * static_cast<size_t>(S) * E, 256);      // bias partials
  }
  if (mf) {
    b += align_up(sizeof(uint16_t) * static_cast<size_t>(T) * route_bwd_ld3(E), 256);  // dl parts
    b += align_up(sizeof(uint16_t) * static_cast<size_t>(d) * 3 * E, 256);            // W_r parts
  }
  return b;
}

namespace {
// dW_r, dbias and dx from the logit gradients on the matrix cores (see the
// top of the file); p = the workspace past the dlogits buffer
hipError_t launch_route_bwd_mfma(const uint16_t* x, const float* w, int64_t T, int d, int E,
                                 const float* dl, float* dw, float* dbias, uint16_t* dx,
                                 int dx_accumulate, char* p, hipStream_t s) {
  const int64_t chunk = route_bwd_mfma_chunk(T, d, E);
  const int S = static_cast<int>(ceil_div(T, chunk));  // chunks that hold tokens
  const int64_t nw = static_cast<int64_t>(d) * E;
  const int ld3 = route_bwd_ld3(E);
  float* part = dw;
  float* bpart = dbias;
  if (S > 1) {
    part = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * static_cast<size_t>(S) * nw, 256);
    bpart = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * static_cast<size_t>(S) * E, 256);
  }
  uint16_t* dl3 = reinterpret_cast<uint16_t*>(p);
  p += align_up(sizeof(uint16_t) * static_cast<size_t>(T) * ld3, 256);
  uint16_t* w3 = reinterpret_cast<uint16_t*>(p);

  prof_begin(K_ROUTE_SPLIT, s);
  route_split_dl_kernel<<<static_cast<unsigned>(ceil_div(T * ld3, 256)), 256, 0, s>>>(dl, T, E,
                                                                                    ld3, dl3);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (dbias != nullptr) {
    route_dbias_part_kernel<<<dim3(static_cast<unsigned>(ceil_div(E, 64)),
                                   static_cast<unsigned>(S)),
                              64 * DB_WAVES, 0, s>>>(dl, T, E, chunk, bpart);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  prof_end(K_ROUTE_SPLIT, s);
  // part[c] = x_c^T (hi + lo)_c for every token chunk c
  if (hipError_t e = launch_router_dw_mfma(x, dl3, T, d, E, ld3, chunk, part, s); e != hipSuccess)
    return e;
  if (S > 1) {
    prof_begin(K_ROUTE_SPLIT, s);
    const int nb = dbias ? E : 0;
    route_dw_reduce_kernel<<<static_cast<unsigned>(ceil_div(nw + nb, 256)), 256, 0, s>>>(
        part, nw, S, dw, bpart, nb, dbias);
    prof_end(K_ROUTE_SPLIT, s);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  if (dx == nullptr) return hipSuccess;
  prof_begin(K_ROUTE_SPLIT, s);
  route_split_w_kernel<<<static_cast<unsigned>(ceil_div(3 * nw, 256)), 256, 0, s>>>(w, d, E, w3);
  prof_end(K_ROUTE_SPLIT, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  // dx [+]= dl3 w3 over the 3E columns, rounded to bf16 once
  return launch_router_dx_mfma(dl3, w3, T, d, E, ld3, dx_accumulate, dx, s);
}
}  // namespace

hipError_t launch_route_bwd(const uint16_t* x, const float* w, const float* logits,
                            const int32_t* idx, const float* gate, const float* dgate,
                            int64_t T, int d, int E, int k, int renorm, float* dw, float* dbias,
                            uint16_t* dx, int dx_accumulate, float* dlogits, void* ws,
                            hipStream_t s) {
  char* p = static_cast<char*>(ws);
  float* dl = dlogits;
  if (dl == nullptr) {
    dl = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * static_cast<size_t>(T) * E, 256);
  }
  const int64_t nw = static_cast<int64_t>(d) * E;
  if (T == 0) {  // no tokens: the weight and bias gradients are exact zeros
    route_zero_kernel<<<static_cast<unsigned>(ceil_div(nw, 256)), 256, 0, s>>>(dw, nw);
    if (dbias) route_zero_kernel<<<static_cast<unsigned>(ceil_div(E, 256)), 256, 0, s>>>(dbias, E);
    return hipGetLastError();
  }
  const unsigned g1 = static_cast<unsigned>(ceil_div(T, 4));
  prof_begin(K_ROUTE_DLOGITS, s);
  if (E <= 64)
    route_dlogits_kernel<1><<<g1, 256, 0, s>>>(logits, idx, gate, dgate, T, E, k, renorm, dl);
  else if (E <= 128)
    route_dlogits_kernel<2><<<g1, 256, 0, s>>>(logits, idx, gate, dgate, T, E, k, renorm, dl);
  else if (E <= 256)
    route_dlogits_kernel<4><<<g1, 256, 0, s>>>(logits, idx, gate, dgate, T, E, k, renorm, dl);
  else if (E <= 512)
    route_dlogits_kernel<8><<<g1, 256, 0, s>>>(logits, idx, gate, dgate, T, E, k, renorm, dl);
  else
    route_dlogits_kernel<16><<<g1, 256, 0, s>>>(logits, idx, gate, dgate, T, E, k, renorm, dl);
  prof_end(K_ROUTE_DLOGITS, s);
  hipError_t err = hipGetLastError();
  if (err != hipSuccess) return err;

  if (route_bwd_mfma(T, d, E))
    return launch_route_bwd_mfma(x, w, T, d, E, dl, dw, dbias, dx, dx_accumulate, p, s);
  const int S = route_bwd_chunks(T, d, E);
  const int64_t chunk = ceil_div(T, S);
  float* part = dw;
  float* bpart = dbias;
  if (S > 1) {
    part = reinterpret_cast<float*>(p);
    p += align_up(sizeof(float) * static_cast<size_t>(S) * d * E, 256);
    bpart = dbias ? reinterpret_cast<float*>(p) : nullptr;
  }
  prof_begin(K_ROUTE_DW, s);
  route_dw_kernel<<<dim3(static_cast<unsigned>(ceil_div(d, RB_J)),
                         static_cast<unsigned>(ceil_div(E, RB_E)), static_cast<unsigned>(S)),
                    256, 0, s>>>(x, dl, T, d, E, chunk, part, bpart);
  if (S > 1) {
    const int nb = dbias ? E : 0;
    route_dw_reduce_kernel<<<static_cast<unsigned>(ceil_div(nw + nb, 256)), 256, 0, s>>>(
        part, nw, S, dw, bpart, nb, dbias);
  }
  prof_end(K_ROUTE_DW, s);
  err = hipGetLastError();
  if (err != hipSuccess || dx == nullptr) return err;

  prof_begin(K_ROUTE_DX, s);
  route_dx_kernel<<<dim3(static_cast<unsigned>(ceil_div(T, RX_T)),
                         static_cast<unsigned>(ceil_div(d, RX_J))),
                    256, 0, s>>>(dl, w, T, d, E, dx_accumulate, dx);
  prof_end(K_ROUTE_DX, s);
  return hipGetLastError();
}

}  // namespace moe
