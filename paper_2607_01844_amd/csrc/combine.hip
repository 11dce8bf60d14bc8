// Weighted combination of expert outputs and its backward (gfx950).
//
// One wave per token; each lane moves 16 bytes (8 bf16) per row and step, so
// a wave reads or writes 1 KiB contiguous per instruction.  The k source
// rows of a token are loaded before they are summed (memory-level
// parallelism), and the sum runs over the slots in ascending order in fp32.
#include "common.h"

namespace moe {
namespace {

__device__ __forceinline__ void unpack8(const uint4& v, float* f) {
  f[0] = bf16_lo(v.x); f[1] = bf16_hi(v.x);
  f[2] = bf16_lo(v.y); f[3] = bf16_hi(v.y);
  f[4] = bf16_lo(v.z); f[5] = bf16_hi(v.z);
  f[6] = bf16_lo(v.w); f[7] = bf16_hi(v.w);
}
__device__ __forceinline__ uint4 pack8(const float* f) {
  return make_uint4(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]), pack_bf16x2(f[4], f[5]),
                    pack_bf16x2(f[6], f[7]));
}

template <int KMAX>
__global__ __launch_bounds__(256) void combine_kernel(const uint16_t* __restrict__ y,
                                                      const int32_t* __restrict__ dst,
                                                      const float* __restrict__ gate, int64_t T,
                                                      int d, int k, uint16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int myp = -1;
  float myg = 0.0f;
  if (lane < k) {
    myp = dst[t * k + lane];
    myg = gate ? gate[t * k + lane] : 1.0f;
  }
  int ps[KMAX];
  float gs[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    ps[i] = __shfl(myp, i, 64);
    gs[i] = __shfl(myg, i, 64);
  }
  const int nch = d >> 3;
  uint4* o = reinterpret_cast<uint4*>(out + t * d);
  for (int c = lane; c < nch; c += 64) {
    uint4 v[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
      if (i < k && ps[i] >= 0)
        v[i] = reinterpret_cast<const uint4*>(y + static_cast<int64_t>(ps[i]) * d)[c];
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      if (i < k && ps[i] >= 0) {
        float f[8];
        unpack8(v[i], f);
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += gs[i] * f[q];
      }
    }
    o[c] = pack8(acc);
  }
}

template <int KMAX>
__global__ __launch_bounds__(256) void combine_bwd_kernel(const uint16_t* __restrict__ dout,
                                                          const uint16_t* __restrict__ y,
                                                          const int32_t* __restrict__ dst,
                                                          const float* __restrict__ gate,
                                                          int64_t T, int d, int k,
                                                          uint16_t* __restrict__ dy_perm,
                                                          float* __restrict__ dgate) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  int myp = -1;
  float myg = 0.0f;
  if (lane < k) {
    myp = dst[t * k + lane];
    myg = gate ? gate[t * k + lane] : 1.0f;
  }
  int ps[KMAX];
  float gs[KMAX];
  float part[KMAX];
#pragma unroll
  for (int i = 0; i < KMAX; ++i) {
    ps[i] = __shfl(myp, i, 64);
    gs[i] = __shfl(myg, i, 64);
    part[i] = 0.0f;
  }
  const int nch = d >> 3;
  const uint4* src = reinterpret_cast<const uint4*>(dout + t * d);
  for (int c = lane; c < nch; c += 64) {
    float g[8];
    unpack8(src[c], g);
    uint4 v[KMAX];
#pragma unroll
    for (int i = 0; i < KMAX; ++i)
      if (i < k && ps[i] >= 0)
        v[i] = reinterpret_cast<const uint4*>(y + static_cast<int64_t>(ps[i]) * d)[c];
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      if (i < k && ps[i] >= 0) {
        float f[8], s[8];
        unpack8(v[i], f);
        float acc = 0.0f;
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          acc += g[q] * f[q];
          s[q] = gs[i] * g[q];
        }
        part[i] += acc;
        reinterpret_cast<uint4*>(dy_perm + static_cast<int64_t>(ps[i]) * d)[c] = pack8(s);
      }
    }
  }
  if (dgate) {
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      if (i < k) {
        const float s = wave_sum(part[i]);
        if (lane == 0) dgate[t * k + i] = (ps[i] >= 0) ? s : 0.0f;
      }
    }
  }
}

}  // namespace

hipError_t launch_combine(const uint16_t* y, const int32_t* dst, const float* gate, int64_t T,
                          int d, int k, uint16_t* out, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const unsigned grid = static_cast<unsigned>(ceil_div(T, 4));
  prof_begin(K_COMBINE, s);
  if (k <= 2)
    combine_kernel<2><<<grid, 256, 0, s>>>(y, dst, gate, T, d, k, out);
  else if (k <= 4)
    combine_kernel<4><<<grid, 256, 0, s>>>(y, dst, gate, T, d, k, out);
  else if (k <= 8)
    combine_kernel<8><<<grid, 256, 0, s>>>(y, dst, gate, T, d, k, out);
  else
    combine_kernel<16><<<grid, 256, 0, s>>>(y, dst, gate, T, d, k, out);
  prof_end(K_COMBINE, s);
  return hipGetLastError();
}

hipError_t launch_combine_bwd(const uint16_t* dout, const uint16_t* y, const int32_t* dst,
                              const float* gate, int64_t T, int d, int k, uint16_t* dy_perm,
                              float* dgate, hipStream_t s) {
  if (T == 0) return hipSuccess;
  const unsigned grid = static_cast<unsigned>(ceil_div(T, 4));
  prof_begin(K_COMBINE_BWD, s);
  if (k <= 2)
    combine_bwd_kernel<2><<<grid, 256, 0, s>>>(dout, y, dst, gate, T, d, k, dy_perm, dgate);
  else if (k <= 4)
    combine_bwd_kernel<4><<<grid, 256, 0, s>>>(dout, y, dst, gate, T, d, k, dy_perm, dgate);
  else if (k <= 8)
    combine_bwd_kernel<8><<<grid, 256, 0, s>>>(dout, y, dst, gate, T, d, k, dy_perm, dgate);
  else
    combine_bwd_kernel<16><<<grid, 256, 0, s>>>(dout, y, dst, gate, T, d, k, dy_perm, dgate);
  prof_end(K_COMBINE_BWD, s);
  return hipGetLastError();
}

}  // namespace moe
