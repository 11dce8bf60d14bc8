// Weighted combination of expert outputs and its backward (gfx950).
//
// One wave per token; each lane moves 16 bytes (8 bf16) per row and step, so
// a wave reads or writes 1 KiB contiguous per instruction.  The forward
// combination reads a token's k source rows one at a time, 8 KiB of a row at
// once (DRAM-friendly bursts), the next row's loads in flight while the
// current one is summed; the backward loads all k rows of a 1 KiB column
// block before it uses them.  Sums run over the slots in ascending order in
// fp32.
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
  // groups of CH chunks per lane (CH KiB of each source row per wave): the
  // rows are read one at a time, the next row's loads issued before the
  // current row is summed
  constexpr int CH = 8;
  for (int c0 = lane; c0 < nch; c0 += 64 * CH) {
    float acc[CH][8];
#pragma unroll
    for (int j = 0; j < CH; ++j)
#pragma unroll
      for (int q = 0; q < 8; ++q) acc[j][q] = 0.0f;
    uint4 cur[CH], nxt[CH];
    auto load_row = [&](int i, uint4* v) {
      const uint4* r = reinterpret_cast<const uint4*>(y + static_cast<int64_t>(ps[i]) * d);
#pragma unroll
      for (int j = 0; j < CH; ++j)
        if (c0 + 64 * j < nch) v[j] = r[c0 + 64 * j];
    };
    if (0 < k && ps[0] >= 0) load_row(0, cur);
#pragma unroll
    for (int i = 0; i < KMAX; ++i) {
      if (i + 1 < KMAX && i + 1 < k && ps[i + 1] >= 0) load_row(i + 1, nxt);
      if (i < k && ps[i] >= 0) {
#pragma unroll
        for (int j = 0; j < CH; ++j) {
          float f[8];
          unpack8(cur[j], f);
#pragma unroll
          for (int q = 0; q < 8; ++q) acc[j][q] += gs[i] * f[q];
        }
      }
#pragma unroll
      for (int j = 0; j < CH; ++j) cur[j] = nxt[j];
    }
#pragma unroll
    for (int j = 0; j < CH; ++j)
      if (c0 + 64 * j < nch) o[c0 + 64 * j] = pack8(acc[j]);
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
