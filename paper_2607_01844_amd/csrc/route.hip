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

typedef int i32x4r __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_byte;

// Compiler-visible wait for every scalar and LDS load of the wave: after it
// the compiler knows all earlier loads have landed, so the loads issued next
// (the following batch) stay in flight while the current batch is computed.
__device__ __forceinline__ void lgkm_drained() { __builtin_amdgcn_s_waitcnt(0xc07f); }

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane, global -> LDS (lane i writes LDS [lds + 16 i, +16));
// completion is tracked by hand with vmcnt.
__device__ __forceinline__ void w_load_lds16(const i32x4r& rsrc, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// Lane = expert (experts lane + 64 b, b < TE); a wave owns TM tokens, a block
// four waves (4 TM tokens).  Each chunk of KC hidden indices moves to
// LDS with direct-to-LDS loads, NBUF chunks deep: the W_r rows (contiguous in
// the row-major [d][E] array) and the block's token rows for those indices.
// Per batch of 8 indices a lane reads its TE weights and, with one broadcast
// 16-byte read per token, the wave's TM x values; the reads of batch b + 1
// are issued before batch b is computed (two register sets).  TWO: the grid
// has at least two blocks per CU, and the chunk ring is sized so that two
// blocks share a CU's LDS (one wave per SIMD leaves the LDS latency exposed).
template <int TM, int TE, int KC, bool TWO>
__global__ __launch_bounds__(256) void route_logits_kernel(const uint16_t* __restrict__ x,
                                                           const float* __restrict__ w,
                                                           const float* __restrict__ bias,
                                                           int64_t T, int d, int E,
                                                           float* __restrict__ logits) {
  constexpr int EW = 64 * TE;                 // experts covered by one block row
  constexpr int WCH = KC * EW * 4;            // LDS bytes of W_r per chunk (>= KC E 4)
  constexpr int TB = 4 * TM;                  // tokens per block
  constexpr int LPWW = WCH / 1024 / 4;        // 1 KiB loads per wave per chunk: W_r
  constexpr int XPL = 1024 / (KC * 2);        // token rows per 1 KiB x load
  constexpr int LPWX = (TB + 4 * XPL - 1) / (4 * XPL);  //                      x
  constexpr int CHUNK = WCH + LPWX * 4 * 1024;  // W_r rows, then the token rows
  constexpr int LDS_CAP = TWO ? 80 * 1024 : 160 * 1024;
  constexpr int NBUF = 4 * CHUNK <= LDS_CAP ? 4 : 3 * CHUNK <= LDS_CAP ? 3 : 2;
  static_assert(KC % 8 == 0 && WCH % 4096 == 0 && (KC * 2) <= 1024 && 1024 % (KC * 2) == 0 &&
                    NBUF * CHUNK <= LDS_CAP,
                "chunk shape");
  __shared__ __align__(16) char ws[NBUF * CHUNK];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int64_t t0 = static_cast<int64_t>(blockIdx.x) * TB;
  float acc[TM][TE];
#pragma unroll
  for (int a = 0; a < TM; ++a)
#pragma unroll
    for (int b = 0; b < TE; ++b) acc[a][b] = +0.0f;

  auto rsrc = [](const void* p, int64_t bytes) {
    const uint64_t addr = reinterpret_cast<uint64_t>(p);
    i32x4r r;
    r[0] = __builtin_amdgcn_readfirstlane(static_cast<int>(addr & 0xffffffffu));
    r[1] = __builtin_amdgcn_readfirstlane(static_cast<int>((addr >> 32) & 0xffffu));
    r[2] = static_cast<int>(bytes > 0x7ffffff0 ? 0x7ffffff0 : (bytes < 0 ? 0 : bytes));
    r[3] = 0x00020000;
    return r;
  };
  // W_r: chunk c = bytes [c KC E 4, +KC E 4); the loads run over WCH bytes
  // (past the chunk: the next rows or, past the array, zeros), which land
  // beyond the KC E floats that are read.  x: the block's token rows from t0
  // (rows past T read as zeros; their logits are never stored).
  const int64_t wbytes = static_cast<int64_t>(d) * E * 4;
  const i32x4r rw = rsrc(w, wbytes);
  const i32x4r rx = rsrc(x + t0 * d, (T - t0) * d * 2);
  const uint32_t lds0 =
      static_cast<uint32_t>(reinterpret_cast<uintptr_t>((const lds_byte*)(ws)));
  auto issue_chunk = [&](int c) __attribute__((always_inline)) {
    const uint32_t dst = lds0 + (c % NBUF) * CHUNK;
    const int64_t wb = static_cast<int64_t>(c) * KC * E * 4;
#pragma unroll
    for (int i = 0; i < LPWW; ++i) {
      const int q = wv * LPWW + i;
      const int64_t off = wb + q * 1024 + lane * 16;
      w_load_lds16(rw, off < wbytes ? static_cast<uint32_t>(off) : 0x80000000u, dst + q * 1024);
    }
    // x: load q covers token rows XPL q .. XPL q + XPL - 1, KC * 2 bytes each
#pragma unroll
    for (int i = 0; i < LPWX; ++i) {
      const int q = wv * LPWX + i;
      const int r = q * XPL + lane / (KC / 8);   // token row of this lane
      const int j = c * KC + (lane % (KC / 8)) * 8;
      const bool ok = r < TB && j < d;
      w_load_lds16(rx, ok ? static_cast<uint32_t>((static_cast<int64_t>(r) * d + j) * 2) : 0x80000000u,
                   dst + WCH + q * 1024);
    }
  };
  // one batch = 8 hidden indices: the wave's x words and the lane's weights
  uint4 xs[2][TM];
  float wq[2][8][TE];
  auto issue = [&](int slot, const char* cb, int bl) __attribute__((always_inline)) {
    const float* cw = reinterpret_cast<const float*>(cb);
#pragma unroll
    for (int a = 0; a < TM; ++a)
      xs[slot][a] = *reinterpret_cast<const uint4*>(cb + WCH + (wv * TM + a) * (KC * 2) + bl * 16);
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int b = 0; b < TE; ++b) wq[slot][u][b] = cw[(bl * 8 + u) * E + lane + 64 * b];
  };
  auto compute = [&](int slot) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 8; ++u) {
#pragma unroll
      for (int a = 0; a < TM; ++a) {
        const uint4 xv = xs[slot][a];
        const uint32_t pr = u < 2 ? xv.x : u < 4 ? xv.y : u < 6 ? xv.z : xv.w;
        const float xa = (u & 1) ? bf16_hi(pr) : bf16_lo(pr);
#pragma unroll
        for (int b = 0; b < TE; ++b) acc[a][b] = __builtin_fmaf(xa, wq[slot][u][b], acc[a][b]);
      }
    }
  };
  // lanes of experts past E read weights of other experts: harmless, never stored
  const int nch = (d + KC - 1) / KC;
#pragma unroll
  for (int c = 0; c < NBUF - 1; ++c) issue_chunk(c);
  for (int c = 0; c < nch; ++c) {
    wait_vm<(LPWW + LPWX) * (NBUF - 2)>();  // this wave's part of chunk c has landed
    __syncthreads();                         // everyone's part; chunk c - 1 is consumed
    issue_chunk(c + NBUF - 1);               // into chunk c - 1's buffer (zeros past the end)
    const char* cb = ws + (c % NBUF) * CHUNK;
    const int nbl = min(KC, d - c * KC) / 8;  // batches in this chunk
    issue(0, cb, 0);
    for (int bl = 0; bl < nbl; bl += 2) {
      lgkm_drained();  // batch bl has landed
      if (bl + 1 < nbl) issue(1, cb, bl + 1);
      compute(0);
      if (bl + 1 < nbl) {
        lgkm_drained();
        if (bl + 2 < nbl) issue(0, cb, bl + 2);
        compute(1);
      }
    }
  }
  wait_vm<0>();  // the trailing chunk loads (zeros) are done before the block ends
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
// A NaN logit ranks as -inf, so every round picks a valid expert (the
// lowest free index when all free logits are -inf or NaN); gates of such a
// token are unspecified.
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
      const float le = l[e];
      v[i] = le != le ? -__builtin_huge_valf() : le;
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
  // chunk rows: KC * TE a multiple of 16 (whole 4 KiB per chunk buffer)
  constexpr int KC = TE == 1 ? 128 : TE == 2 ? 64 : TE == 4 ? 32 : TE <= 8 ? 16 : 8;
  const int64_t grid = ceil_div(T, 4 * TM);
  prof_begin(K_ROUTE_LOGITS, s);
  if (grid >= 2 * static_cast<int64_t>(device_cus()))
    route_logits_kernel<TM, TE, KC, true><<<static_cast<unsigned>(grid), 256, 0, s>>>(
        x, w, bias, T, d, E, logits);
  else
    route_logits_kernel<TM, TE, KC, false><<<static_cast<unsigned>(grid), 256, 0, s>>>(
        x, w, bias, T, d, E, logits);
  prof_end(K_ROUTE_LOGITS, s);
  return hipGetLastError();
}

// Tokens per wave: about two blocks per CU (T / 2048 tokens per wave,
// rounded down to 8, 4, 2 or 1), so that two waves share each SIMD while
// every block still reads W_r for as many tokens as the chip's share allows,
// with at most 64 accumulators per lane (TM * TE <= 64).
template <int TE>
hipError_t pick_logits(const uint16_t* x, const float* w, const float* bias, int64_t T, int d,
                       int E, float* logits, hipStream_t s) {
  if constexpr (8 * TE <= 64)
    if (T >= 16 * 1024) return run_logits<8, TE>(x, w, bias, T, d, E, logits, s);
  if constexpr (4 * TE <= 64)
    if (T >= 8 * 1024) return run_logits<4, TE>(x, w, bias, T, d, E, logits, s);
  if (T >= 4 * 1024) return run_logits<2, TE>(x, w, bias, T, d, E, logits, s);
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
