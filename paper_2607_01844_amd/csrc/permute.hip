// Permutation of token-expert assignments into per-expert segments (gfx950).
//
// A stable counting sort by local expert id over assignments a = t*k + i:
//   1. count: per block of CH assignments, per-expert counts (LDS atomics;
//      only counts, so their order does not matter).
//   2. scan: one workgroup turns the block counts into expert_offsets and a
//      per-(block, expert) base.
//   3. rank: each wave walks its slice of the block in order; lanes of one
//      64-assignment step that share an expert are found with ballots over
//      the bits of the expert id, and ranked by lane order (popcount of the
//      lower lanes).  Positions never depend on atomic return order.
//   4. gather: one wave per token reads x[t] once and writes it to each of
//      the token's local rows.
#include <mutex>

#include "common.h"

namespace moe {

// Scratch of the allocation-free permutation (moe_permute_noalloc): the
// per-block expert counts and bases, in a static device array that every
// GPU the library runs on holds until the process ends.  In host code the
// array's name is only a host-side stand-in, never a device address: the
// device address comes from hipGetSymbolAddress, looked up once per device
// with that device current.  Every call on one GPU shares that GPU's copy,
// so calls that overlap on one GPU (different streams) race.  The kernels
// write every scratch word they read, so nothing is cleared between calls.
static __device__ __align__(256) char scratch[MOE_PERMUTE_NOALLOC_MAX_BYTES];

namespace {

constexpr int CH = 4096;          // assignments per count/rank block
constexpr int RANK_WAVES = 4;     // 256 threads
constexpr int PER_WAVE = CH / RANK_WAVES;
constexpr int RANK_ITERS = PER_WAVE / 64;

__global__ __launch_bounds__(256) void perm_count_kernel(const int32_t* __restrict__ idx,
                                                         int64_t A, int E, int e_begin,
                                                         int E_loc, int32_t* __restrict__ blk_loc,
                                                         int32_t* __restrict__ blk_glob) {
  extern __shared__ int sh[];
  int* hl = sh;
  int* hg = sh + E_loc;
  for (int i = threadIdx.x; i < E_loc + E; i += 256) sh[i] = 0;
  __syncthreads();
  const int64_t a0 = static_cast<int64_t>(blockIdx.x) * CH;
  const int64_t a1 = min(a0 + CH, A);
  for (int64_t a = a0 + threadIdx.x; a < a1; a += 256) {
    const int e = idx[a];
    if (static_cast<unsigned>(e) < static_cast<unsigned>(E)) {
      atomicAdd(&hg[e], 1);
      const int el = e - e_begin;
      if (static_cast<unsigned>(el) < static_cast<unsigned>(E_loc)) atomicAdd(&hl[el], 1);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < E_loc; i += 256)
    blk_loc[static_cast<int64_t>(blockIdx.x) * E_loc + i] = hl[i];
  for (int i = threadIdx.x; i < E; i += 256)
    blk_glob[static_cast<int64_t>(blockIdx.x) * E + i] = hg[i];
}

// One workgroup of 1024 threads (E_loc, E <= 1024).
__global__ __launch_bounds__(1024) void perm_scan_kernel(const int32_t* __restrict__ blk_loc,
                                                         const int32_t* __restrict__ blk_glob,
                                                         int nb, int E, int E_loc,
                                                         int32_t* __restrict__ pre,
                                                         int32_t* __restrict__ offsets,
                                                         int32_t* __restrict__ counts_global) {
  __shared__ int tot[1024];
  __shared__ int wsum[16];
  const int e = threadIdx.x;
  // the walks over the nb blocks below load 8 blocks' values before using
  // them: a dependent load per block would cost one memory round trip each
  constexpr int U = 8;
  int run = 0;
  if (e < E_loc) {
    int b = 0;
    for (; b + U <= nb; b += U) {
      int c[U];
#pragma unroll
      for (int u = 0; u < U; ++u) c[u] = blk_loc[static_cast<int64_t>(b + u) * E_loc + e];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        pre[static_cast<int64_t>(b + u) * E_loc + e] = run;
        run += c[u];
      }
    }
    for (; b < nb; ++b) {
      const int c = blk_loc[static_cast<int64_t>(b) * E_loc + e];
      pre[static_cast<int64_t>(b) * E_loc + e] = run;
      run += c;
    }
  }
  // exclusive scan of the per-expert totals over e: wave scans + wave sums
  const int lane = e & 63, w = e >> 6;
  int incl = run;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(incl, o, 64);
    if (lane >= o) incl += y;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int wbase = 0;
  for (int i = 0; i < w; ++i) wbase += wsum[i];
  const int excl = wbase + incl - run;
  tot[e] = excl;
  if (e < E_loc) {
    offsets[e] = excl;
    int b = 0;
    for (; b + U <= nb; b += U) {
      int v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = pre[static_cast<int64_t>(b + u) * E_loc + e];
#pragma unroll
      for (int u = 0; u < U; ++u) pre[static_cast<int64_t>(b + u) * E_loc + e] = v[u] + excl;
    }
    for (; b < nb; ++b) pre[static_cast<int64_t>(b) * E_loc + e] += excl;
  }
  if (e == E_loc - 1) offsets[E_loc] = excl + run;
  if (counts_global && e < E) {
    int s = 0, b = 0;
    for (; b + U <= nb; b += U) {
      int v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) v[u] = blk_glob[static_cast<int64_t>(b + u) * E + e];
#pragma unroll
      for (int u = 0; u < U; ++u) s += v[u];
    }
    for (; b < nb; ++b) s += blk_glob[static_cast<int64_t>(b) * E + e];
    counts_global[e] = s;
  }
}

__global__ __launch_bounds__(256) void perm_rank_kernel(const int32_t* __restrict__ idx,
                                                        int64_t A, int e_begin, int E_loc,
                                                        int nbits,
                                                        const int32_t* __restrict__ pre,
                                                        int32_t* __restrict__ row_src,
                                                        int32_t* __restrict__ dst) {
  extern __shared__ int cnt[];  // [RANK_WAVES][E_loc]
  for (int i = threadIdx.x; i < RANK_WAVES * E_loc; i += 256) cnt[i] = 0;
  __syncthreads();
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int* mycnt = cnt + w * E_loc;
  const int64_t base = static_cast<int64_t>(blockIdx.x) * CH + w * PER_WAVE;
  const uint64_t lt = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  int rk[RANK_ITERS];
  int els[RANK_ITERS];
#pragma unroll
  for (int it = 0; it < RANK_ITERS; ++it) {
    const int64_t a = base + it * 64 + lane;
    int el = E_loc;  // sentinel: not local / past the end
    if (a < A) {
      const int v = idx[a] - e_begin;
      if (static_cast<unsigned>(v) < static_cast<unsigned>(E_loc)) el = v;
    }
    uint64_t same = ~0ull;
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (el >> b) & 1;
      const uint64_t bal = __ballot(bit);
      same &= bit ? bal : ~bal;
    }
    int r = 0;
    if (el != E_loc) {
      const int prev = mycnt[el];
      r = prev + __popcll(same & lt);
      if ((same >> lane) == 1ull) mycnt[el] = prev + __popcll(same);
    }
    rk[it] = r;
    els[it] = el;
  }
  __syncthreads();
  // per expert: exclusive offsets of the 4 waves of this block
  for (int e = threadIdx.x; e < E_loc; e += 256) {
    int run = 0;
#pragma unroll
    for (int ww = 0; ww < RANK_WAVES; ++ww) {
      const int c = cnt[ww * E_loc + e];
      cnt[ww * E_loc + e] = run;
      run += c;
    }
  }
  __syncthreads();
  const int32_t* bpre = pre + static_cast<int64_t>(blockIdx.x) * E_loc;
#pragma unroll
  for (int it = 0; it < RANK_ITERS; ++it) {
    const int64_t a = base + it * 64 + lane;
    if (a >= A) continue;
    const int el = els[it];
    if (el == E_loc) {
      dst[a] = -1;
    } else {
      const int p = bpre[el] + mycnt[el] + rk[it];
      dst[a] = p;
      row_src[p] = static_cast<int32_t>(a);
    }
  }
}

__global__ __launch_bounds__(256) void perm_gather_kernel(const uint16_t* __restrict__ x,
                                                          const int32_t* __restrict__ dst,
                                                          int64_t T, int d, int k,
                                                          uint16_t* __restrict__ x_perm) {
  const int lane = threadIdx.x & 63;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6);
  if (t >= T) return;
  const int my = (lane < k) ? dst[t * k + lane] : -1;
  if (__ballot(my >= 0) == 0ull) return;
  int ps[MOE_MAX_K];
#pragma unroll
  for (int i = 0; i < MOE_MAX_K; ++i) ps[i] = __shfl(my, i, 64);
  const uint4* src = reinterpret_cast<const uint4*>(x + t * d);
  const int nch = d >> 3;
  for (int c0 = lane; c0 < nch; c0 += 4 * 64) {
    uint4 v[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = c0 + u * 64;
      if (c < nch) v[u] = src[c];
    }
#pragma unroll
    for (int i = 0; i < MOE_MAX_K; ++i) {
      if (i >= k) break;
      if (ps[i] < 0) continue;
      uint4* out = reinterpret_cast<uint4*>(x_perm + static_cast<int64_t>(ps[i]) * d);
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = c0 + u * 64;
        if (c < nch) out[c] = v[u];
      }
    }
  }
}

// Rows [r0, r0 + rc) of the permuted order (consecutive experts, the first
// and last possibly in part) as a layer of their own: their expert offsets,
// offsets_c[e] = clamp(offsets[e] - r0, 0, rc) for e = 0..E_loc, and their
// rows of x (row i from token row_src[r0 + i] / k), up to the last filled
// row.  One wave per row, 16 bytes per lane.
__global__ __launch_bounds__(256) void perm_chunk_rows_kernel(
    const uint16_t* __restrict__ x, const int32_t* __restrict__ row_src,
    const int32_t* __restrict__ offsets, int E_loc, int64_t r0, int64_t rc, int d, int k,
    int32_t* __restrict__ offsets_c, uint16_t* __restrict__ x_perm_c) {
  auto clamp_rows = [&](int32_t o) {
    return static_cast<int32_t>(min(max(static_cast<int64_t>(o) - r0, int64_t{0}), rc));
  };
  if (blockIdx.x == 0) {
    for (int e = threadIdx.x; e <= E_loc; e += blockDim.x) offsets_c[e] = clamp_rows(offsets[e]);
  }
  const int64_t m = clamp_rows(offsets[E_loc]);
  const int lane = threadIdx.x & 63;
  const int nch = d >> 3;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * 4 + (threadIdx.x >> 6); i < m;
       i += static_cast<int64_t>(gridDim.x) * 4) {
    const int64_t t = row_src[r0 + i] / k;
    const uint4* src = reinterpret_cast<const uint4*>(x + t * d);
    uint4* out = reinterpret_cast<uint4*>(x_perm_c + i * d);
    for (int c = lane; c < nch; c += 64) out[c] = src[c];
  }
}

struct PermWs {
  int32_t* blk_loc;
  int32_t* blk_glob;
  int32_t* pre;
};

PermWs carve(void* ws, int nb, int E, int E_loc) {
  char* p = static_cast<char*>(ws);
  PermWs w;
  w.blk_loc = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * static_cast<size_t>(nb) * E_loc, 256);
  w.blk_glob = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * static_cast<size_t>(nb) * E, 256);
  w.pre = reinterpret_cast<int32_t*>(p);
  return w;
}

}  // namespace

size_t permute_ws_bytes(int64_t T, int E, int k, int E_loc) {
  const int64_t nb = ceil_div(T * k, CH);
  return align_up(sizeof(int32_t) * nb * E_loc, 256) + align_up(sizeof(int32_t) * nb * E, 256) +
         align_up(sizeof(int32_t) * nb * E_loc, 256) + 256;
}

hipError_t launch_permute(const uint16_t* x, const int32_t* idx, int64_t T, int d, int E, int k,
                          int e_begin, int E_loc, int32_t* offsets, int32_t* counts_global,
                          int32_t* row_src, int32_t* dst, uint16_t* x_perm, void* ws,
                          hipStream_t s) {
  const int64_t A = T * k;
  const int nb = static_cast<int>(ceil_div(A, CH));
  PermWs w = carve(ws, nb, E, E_loc);
  if (nb > 0) {
    prof_begin(K_PERM_COUNT, s);
    perm_count_kernel<<<nb, 256, sizeof(int) * (E_loc + E), s>>>(idx, A, E, e_begin, E_loc,
                                                                 w.blk_loc, w.blk_glob);
    prof_end(K_PERM_COUNT, s);
    if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  }
  prof_begin(K_PERM_SCAN, s);
  perm_scan_kernel<<<1, 1024, 0, s>>>(w.blk_loc, w.blk_glob, nb, E, E_loc, w.pre, offsets,
                                      counts_global);
  prof_end(K_PERM_SCAN, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (nb == 0) return hipSuccess;
  int nbits = 0;
  while ((1 << nbits) <= E_loc) ++nbits;  // ids 0..E_loc (E_loc = sentinel)
  prof_begin(K_PERM_RANK, s);
  perm_rank_kernel<<<nb, 256, sizeof(int) * RANK_WAVES * E_loc, s>>>(idx, A, e_begin, E_loc,
                                                                     nbits, w.pre, row_src, dst);
  prof_end(K_PERM_RANK, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (x_perm == nullptr) return hipSuccess;  // the index only
  prof_begin(K_PERM_GATHER, s);
  perm_gather_kernel<<<static_cast<unsigned>(ceil_div(T, 4)), 256, 0, s>>>(x, dst, T, d, k,
                                                                           x_perm);
  prof_end(K_PERM_GATHER, s);
  return hipGetLastError();
}

hipError_t launch_chunk_rows(const uint16_t* x, const int32_t* row_src, const int32_t* offsets,
                             int E_loc, int64_t r0, int64_t rc, int d, int k, int32_t* offsets_c,
                             uint16_t* x_perm_c, hipStream_t s) {
  const unsigned grid = static_cast<unsigned>(std::max<int64_t>(1, std::min<int64_t>(ceil_div(rc, 4), 1 << 16)));
  prof_begin(K_PERM_GATHER, s);
  perm_chunk_rows_kernel<<<grid, 256, 0, s>>>(x, row_src, offsets, E_loc, r0, rc, d, k, offsets_c,
                                              x_perm_c);
  prof_end(K_PERM_GATHER, s);
  return hipGetLastError();
}

namespace {
constexpr int kScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kScratchDevices] = {};

// the current device's address of `scratch` (looked up on first use)
hipError_t scratch_address(void** out) {
  int dev = -1;
  if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return e;
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    if (hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)); e != hipSuccess) return e;
    if (ptr == nullptr) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}
}  // namespace

hipError_t launch_permute_noalloc(const uint16_t* x, const int32_t* idx, int64_t T, int d, int E,
                                  int k, int e_begin, int E_loc, int32_t* offsets,
                                  int32_t* counts_global, int32_t* row_src, int32_t* dst,
                                  uint16_t* x_perm, hipStream_t s) {
  void* ws = nullptr;
  if (hipError_t e = scratch_address(&ws); e != hipSuccess) return e;
  return launch_permute(x, idx, T, d, E, k, e_begin, E_loc, offsets, counts_global, row_src, dst,
                        x_perm, ws, s);
}

hipError_t launch_gather(const uint16_t* x, const int32_t* dst, int64_t T, int d, int k,
                         uint16_t* x_perm, hipStream_t s) {
  if (T == 0) return hipSuccess;
  prof_begin(K_PERM_GATHER, s);
  perm_gather_kernel<<<static_cast<unsigned>(ceil_div(T, 4)), 256, 0, s>>>(x, dst, T, d, k,
                                                                           x_perm);
  prof_end(K_PERM_GATHER, s);
  return hipGetLastError();
}

}  // namespace moe
