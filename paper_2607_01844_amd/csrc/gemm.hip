// Grouped SwiGLU expert GEMMs on gfx950 (bf16 MFMA, fp32 accumulation).
//
// Every GEMM of the expert FFN (forward gate/up and down, data gradients,
// weight gradients) is one instance of a single macro-tile kernel:
//   * 256 threads = 4 waves in a 2 x 2 grid; the block computes a 256 x 256
//     tile of C^T (rows = output columns n, cols = output rows m) with
//     v_mfma_f32_32x32x16_bf16, so each lane ends up holding four consecutive
//     output columns and stores 8 bytes at a time.
//   * K steps of 64; both operand tiles live in LDS as [256 rows][64 k] bf16
//     with a 16-byte-chunk XOR swizzle (conflict-free ds_read_b128 for the
//     MFMA fragments and conflict-free writes); two LDS stages (128 KiB), the
//     next K step's global loads are in flight while the current one runs.
//   * Operands stored K-contiguous are copied straight to LDS; operands
//     stored with the output index contiguous (weights in the forward pass,
//     everything in the weight gradients) are loaded as 8 x 8 blocks and
//     transposed in registers with v_perm_b32 before the LDS write.
//   * Variable-size expert segments: a tiny scheduler kernel turns
//     expert_offsets into per-expert tile counts on the device (no host
//     synchronisation, no padding to a capacity).  Row tails are masked; an
//     expert without rows gets no forward tiles and zero weight gradients.
//   * XCD-aware order: gfx950 hands consecutive workgroups to its 8 XCDs in
//     turn, and each XCD has its own L2.  Logical tiles are laid out so each
//     XCD runs a contiguous range of them, and inside one expert the row
//     tiles of one weight tile are adjacent: they share that weight tile in
//     the same L2, so each weight byte comes from HBM about once.
#include "common.h"

namespace moe {
namespace {

constexpr int BM = 256;      // tile rows on the operand-A side (m)
constexpr int BN = 256;      // tile rows on the operand-B side (n)
constexpr int BK = 64;
constexpr int TILE_BYTES = 256 * BK * 2;  // one operand tile in LDS (32 KiB)
constexpr int NXCD = 8;

enum Mode {
  FWD_GATE_UP = 0,  // Hg, Hu, A  = X Wg, X Wu, silu(Hg) Hu       (dual B, K = d)
  FWD_DOWN,         // Y = A Wd                                    (K = f)
  DGRAD_DOWN,       // dA = dY Wd^T -> dHg, dHu, A                 (K = d)
  DGRAD_GATE_UP,    // dX = dHg Wg^T + dHu Wu^T                    (K = 2f)
  WGRAD_GATE_UP,    // dWg, dWu = X^T dHg, X^T dHu                 (dual B, K = n_e)
  WGRAD_DOWN        // dWd = A^T dY                                (K = n_e)
};

// byte offset of 16-byte chunk `c` (k = 8c..8c+7) of tile row `r`
__device__ __forceinline__ int lds_off(int r, int c) {
  return r * (BK * 2) + ((c ^ ((r ^ (r >> 3)) & 7)) << 4);
}

// ---------------------------------------------------------------- loaders
// K-contiguous operand: element (r, k) at b0[r*ld + k] for k < ksplit and at
// b1[r*ld + k - ksplit] otherwise; r < rows and k < kmax are valid, the rest
// reads as zero.  256 rows x 64 k per step, 8 chunks of 16 bytes per thread.
struct KLoader {
  const uint16_t* b0;
  const uint16_t* b1;
  int64_t ld;
  int rows, ksplit, kmax;
  uint4 v[8];

  __device__ __forceinline__ void load(int kt) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + 256 * i;
      const int r = q >> 3, c = q & 7;
      const int k = kt * BK + c * 8;
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (r < rows && k < kmax) {
        const uint16_t* p = (k < ksplit) ? b0 + r * ld + k : b1 + r * ld + (k - ksplit);
        val = *reinterpret_cast<const uint4*>(p);
      }
      v[i] = val;
    }
  }
  __device__ __forceinline__ void store(char* tile) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int q = tid + 256 * i;
      *reinterpret_cast<uint4*>(tile + lds_off(q >> 3, q & 7)) = v[i];
    }
  }
};

// Transposed operand: element (r, k) at b[k*ld + r] (r contiguous).  Tile
// rows r < split come from b0 (column r), rows r >= split from b1 (column
// r - split); columns >= rmax and k >= kmax read as zero.  Each thread loads
// an 8 (k) x 8 (r) block and writes 8 rows of 8 k to LDS.
struct TLoader {
  const uint16_t* b0;
  const uint16_t* b1;
  int64_t ld;
  int split, rmax, kmax;
  uint4 v[8];

  __device__ __forceinline__ void load(int kt) {
    const int tid = threadIdx.x;
    const int kb = tid >> 5, nb = tid & 31;
    const int c0 = nb * 8;
    const uint16_t* src = (c0 < split) ? b0 + c0 : b1 + (c0 - split);
    const int col = (c0 < split) ? c0 : c0 - split;
    const bool cok = col < rmax;
    const int k0 = kt * BK + kb * 8;
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      uint4 val = make_uint4(0u, 0u, 0u, 0u);
      if (cok && k0 + r < kmax) val = *reinterpret_cast<const uint4*>(src + (k0 + r) * ld);
      v[r] = val;
    }
  }
  __device__ __forceinline__ void store(char* tile) const {
    const int tid = threadIdx.x;
    const int kb = tid >> 5, nb = tid & 31;
    const uint32_t* w = reinterpret_cast<const uint32_t*>(v);  // w[4*k + j] = cols 2j, 2j+1
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      uint4 even, odd;
      uint32_t* pe = reinterpret_cast<uint32_t*>(&even);
      uint32_t* po = reinterpret_cast<uint32_t*>(&odd);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t lo = w[4 * (2 * i) + j], hi = w[4 * (2 * i + 1) + j];
        pe[i] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
        po[i] = __builtin_amdgcn_perm(hi, lo, 0x07060302u);
      }
      *reinterpret_cast<uint4*>(tile + lds_off(nb * 8 + 2 * j, kb)) = even;
      *reinterpret_cast<uint4*>(tile + lds_off(nb * 8 + 2 * j + 1, kb)) = odd;
    }
  }
};

struct GemmArgs {
  // inputs
  const uint16_t* x_perm;   // [cap][d]
  const uint16_t* wg;       // [E_loc][d][f]
  const uint16_t* wu;
  const uint16_t* wd;       // [E_loc][f][d]
  const uint16_t* hg_in;    // [cap][f]
  const uint16_t* hu_in;
  const uint16_t* act_in;   // [cap][f]
  const uint16_t* dy;       // [cap][d]
  const uint16_t* dhg_in;   // [cap][f]
  const uint16_t* dhu_in;
  const int32_t* offsets;   // [E_loc+1]
  const int32_t* mt_start;  // [E_loc+1] prefix of per-expert row-tile counts
  const int32_t* lpt;       // [E_loc] experts by rows, descending
  // outputs
  uint16_t* hg;
  uint16_t* hu;
  uint16_t* act;
  uint16_t* y;
  uint16_t* dhg;
  uint16_t* dhu;
  uint16_t* dx;
  uint16_t* dwg;
  uint16_t* dwu;
  uint16_t* dwd;
  int E_loc, d, f;
  int NT;  // column tiles per row tile
  int MT;  // row tiles per expert (weight-gradient modes)
};

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ uint2 pack4(float a, float b, float c, float d) {
  return make_uint2(pack_bf16x2(a, b), pack_bf16x2(c, d));
}

template <int MODE>
__global__ __launch_bounds__(256, 1) void grouped_gemm_kernel(GemmArgs g) {
  __shared__ __align__(16) char lds[2 * 2 * TILE_BYTES];
  constexpr bool WGRAD = (MODE == WGRAD_GATE_UP || MODE == WGRAD_DOWN);
  constexpr bool DUAL = (MODE == FWD_GATE_UP || MODE == WGRAD_GATE_UP);

  // ------------------------------------------------------------ tile pick
  int e, m0, n0, seg, ne;
  const int b = blockIdx.x;
  const int xcd = b % NXCD, slot = b / NXCD;
  if constexpr (!WGRAD) {
    const int total = g.mt_start[g.E_loc] * g.NT;
    const int per = (total + NXCD - 1) / NXCD;
    const int L = xcd * per + slot;
    if (slot >= per || L >= total) return;
    int lo = 0, hi = g.E_loc;
    while (hi - lo > 1) {
      const int mid = (lo + hi) >> 1;
      if (g.mt_start[mid] * g.NT <= L) lo = mid; else hi = mid;
    }
    e = lo;
    const int mt_e = g.mt_start[e + 1] - g.mt_start[e];
    const int local = L - g.mt_start[e] * g.NT;
    const int nt = local / mt_e, mt = local % mt_e;
    seg = g.offsets[e];
    ne = g.offsets[e + 1] - seg;
    m0 = mt * BM;
    n0 = nt * (DUAL ? BN / 2 : BN);
  } else {
    const int per_e = g.MT * g.NT;
    const int rank = xcd + NXCD * (slot / per_e);
    if (rank >= g.E_loc) return;
    e = g.lpt[rank];
    const int local = slot % per_e;
    const int mt = local / g.NT, nt = local % g.NT;
    seg = g.offsets[e];
    ne = g.offsets[e + 1] - seg;
    m0 = mt * BM;
    n0 = nt * (DUAL ? BN / 2 : BN);
  }
  const int d = g.d, f = g.f;
  const int64_t wdf = static_cast<int64_t>(d) * f;

  // ------------------------------------------------------- operand setup
  // A side = rows m of the output, B side = columns n of the output.
  using ALoader = typename std::conditional<WGRAD, TLoader, KLoader>::type;
  using BLoader = typename std::conditional<MODE == DGRAD_DOWN || MODE == DGRAD_GATE_UP,
                                            KLoader, TLoader>::type;
  ALoader la;
  BLoader lb;
  int nk = 0;
  if constexpr (MODE == FWD_GATE_UP) {
    la = KLoader{g.x_perm + (int64_t)(seg + m0) * d, nullptr, d, ne - m0, d, d};
    lb = TLoader{g.wg + e * wdf + n0, g.wu + e * wdf + n0, f, BN / 2, f - n0, d};
    nk = (d + BK - 1) / BK;
  } else if constexpr (MODE == FWD_DOWN) {
    la = KLoader{g.act_in + (int64_t)(seg + m0) * f, nullptr, f, ne - m0, f, f};
    lb = TLoader{g.wd + e * wdf + n0, nullptr, d, BN, d - n0, f};
    nk = (f + BK - 1) / BK;
  } else if constexpr (MODE == DGRAD_DOWN) {
    la = KLoader{g.dy + (int64_t)(seg + m0) * d, nullptr, d, ne - m0, d, d};
    lb = KLoader{g.wd + e * wdf + (int64_t)n0 * d, nullptr, d, f - n0, d, d};
    nk = (d + BK - 1) / BK;
  } else if constexpr (MODE == DGRAD_GATE_UP) {
    la = KLoader{g.dhg_in + (int64_t)(seg + m0) * f, g.dhu_in + (int64_t)(seg + m0) * f, f,
                 ne - m0, f, 2 * f};
    lb = KLoader{g.wg + e * wdf + (int64_t)n0 * f, g.wu + e * wdf + (int64_t)n0 * f, f, d - n0,
                 f, 2 * f};
    nk = (2 * f + BK - 1) / BK;
  } else if constexpr (MODE == WGRAD_GATE_UP) {
    la = TLoader{g.x_perm + (int64_t)seg * d + m0, nullptr, d, BM, d - m0, ne};
    lb = TLoader{g.dhg_in + (int64_t)seg * f + n0, g.dhu_in + (int64_t)seg * f + n0, f, BN / 2,
                 f - n0, ne};
    nk = (ne + BK - 1) / BK;
  } else {  // WGRAD_DOWN
    la = TLoader{g.act_in + (int64_t)seg * f + m0, nullptr, f, BM, f - m0, ne};
    lb = TLoader{g.dy + (int64_t)seg * d + n0, nullptr, d, BN, d - n0, ne};
    nk = (ne + BK - 1) / BK;
  }

  // -------------------------------------------------------------- K loop
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wm = w >> 1, wn = w & 1;
  const int l32 = lane & 31, lh = lane >> 5;
  int arow[4], brow[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    arow[i] = wm * 128 + 32 * i + l32;
    if constexpr (DUAL)
      brow[i] = (i < 2 ? 0 : BN / 2) + wn * 64 + 32 * (i & 1) + l32;
    else
      brow[i] = wn * 128 + 32 * i + l32;
  }

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  if (nk > 0) {
    la.load(0);
    lb.load(0);
    la.store(lds);
    lb.store(lds + TILE_BYTES);
    __syncthreads();
  }
  for (int kt = 0; kt < nk; ++kt) {
    char* cur = lds + (kt & 1) * 2 * TILE_BYTES;
    char* nxt = lds + ((kt + 1) & 1) * 2 * TILE_BYTES;
    const bool more = kt + 1 < nk;
    if (more) {
      la.load(kt + 1);
      lb.load(kt + 1);
    }
    const char* ta = cur;
    const char* tb = cur + TILE_BYTES;
#pragma unroll
    for (int s = 0; s < BK / 16; ++s) {
      bf16x8 af[4], bfr[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(ta + lds_off(arow[i], 2 * s + lh));
#pragma unroll
      for (int j = 0; j < 4; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(tb + lds_off(brow[j], 2 * s + lh));
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = mfma(bfr[j], af[i], acc[i][j]);
    }
    if (more) {
      la.store(nxt);
      lb.store(nxt + TILE_BYTES);
    }
    __syncthreads();
  }

  // ------------------------------------------------------------ epilogue
  // acc[i][j][4q + u]: output row m = arow[i] (tile-relative),
  // output column n = (B-tile row of block j) + 8q + 4*lh + u.
  const int mvalid = WGRAD ? ((MODE == WGRAD_GATE_UP ? d : f) - m0) : (ne - m0);
  static_for<4>([&](auto I) {
    constexpr int i = I;
    const int m = arow[i];
    if (m < mvalid) {
      if constexpr (MODE == FWD_GATE_UP || MODE == WGRAD_GATE_UP) {
        static_for<2>([&](auto J) {
          constexpr int j = J;
          static_for<4>([&](auto Q) {
            constexpr int q = Q;
            const int n = wn * 64 + 32 * j + 8 * q + 4 * lh;  // f index within tile
            if (n0 + n < f) {
              const f32x16& ga = acc[i][j];
              const f32x16& ua = acc[i][j + 2];
              if constexpr (MODE == FWD_GATE_UP) {
                const int64_t o = (int64_t)(seg + m0 + m) * f + n0 + n;
                const uint2 hgb = pack4(ga[4 * q], ga[4 * q + 1], ga[4 * q + 2], ga[4 * q + 3]);
                const uint2 hub = pack4(ua[4 * q], ua[4 * q + 1], ua[4 * q + 2], ua[4 * q + 3]);
                const float g0 = bf16_lo(hgb.x), g1 = bf16_hi(hgb.x);
                const float g2 = bf16_lo(hgb.y), g3 = bf16_hi(hgb.y);
                const float a0 = g0 * sigmoidf_fast(g0) * bf16_lo(hub.x);
                const float a1 = g1 * sigmoidf_fast(g1) * bf16_hi(hub.x);
                const float a2 = g2 * sigmoidf_fast(g2) * bf16_lo(hub.y);
                const float a3 = g3 * sigmoidf_fast(g3) * bf16_hi(hub.y);
                *reinterpret_cast<uint2*>(g.hg + o) = hgb;
                *reinterpret_cast<uint2*>(g.hu + o) = hub;
                *reinterpret_cast<uint2*>(g.act + o) = pack4(a0, a1, a2, a3);
              } else {
                const int64_t o = e * wdf + (int64_t)(m0 + m) * f + n0 + n;
                *reinterpret_cast<uint2*>(g.dwg + o) =
                    pack4(ga[4 * q], ga[4 * q + 1], ga[4 * q + 2], ga[4 * q + 3]);
                *reinterpret_cast<uint2*>(g.dwu + o) =
                    pack4(ua[4 * q], ua[4 * q + 1], ua[4 * q + 2], ua[4 * q + 3]);
              }
            }
          });
        });
      } else {
        static_for<4>([&](auto J) {
          constexpr int j = J;
          static_for<4>([&](auto Q) {
            constexpr int q = Q;
            const int n = wn * 128 + 32 * j + 8 * q + 4 * lh;
            const float c0 = acc[i][j][4 * q], c1 = acc[i][j][4 * q + 1];
            const float c2 = acc[i][j][4 * q + 2], c3 = acc[i][j][4 * q + 3];
            if constexpr (MODE == FWD_DOWN) {
              if (n0 + n < d)
                *reinterpret_cast<uint2*>(g.y + (int64_t)(seg + m0 + m) * d + n0 + n) =
                    pack4(c0, c1, c2, c3);
            } else if constexpr (MODE == DGRAD_GATE_UP) {
              if (n0 + n < d)
                *reinterpret_cast<uint2*>(g.dx + (int64_t)(seg + m0 + m) * d + n0 + n) =
                    pack4(c0, c1, c2, c3);
            } else if constexpr (MODE == WGRAD_DOWN) {
              if (n0 + n < d)
                *reinterpret_cast<uint2*>(g.dwd + e * wdf + (int64_t)(m0 + m) * d + n0 + n) =
                    pack4(c0, c1, c2, c3);
            } else {  // DGRAD_DOWN: SwiGLU backward
              if (n0 + n < f) {
                const int64_t o = (int64_t)(seg + m0 + m) * f + n0 + n;
                const uint2 hgv = *reinterpret_cast<const uint2*>(g.hg_in + o);
                const uint2 huv = *reinterpret_cast<const uint2*>(g.hu_in + o);
                float dg[4], du[4], av[4];
                const float gz[4] = {bf16_lo(hgv.x), bf16_hi(hgv.x), bf16_lo(hgv.y),
                                     bf16_hi(hgv.y)};
                const float uz[4] = {bf16_lo(huv.x), bf16_hi(huv.x), bf16_lo(huv.y),
                                     bf16_hi(huv.y)};
                const float da[4] = {c0, c1, c2, c3};
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                  const float sg = sigmoidf_fast(gz[u]);
                  const float sl = gz[u] * sg;
                  dg[u] = da[u] * uz[u] * (sg + sl * (1.0f - sg));
                  du[u] = da[u] * sl;
                  av[u] = sl * uz[u];
                }
                *reinterpret_cast<uint2*>(g.dhg + o) = pack4(dg[0], dg[1], dg[2], dg[3]);
                *reinterpret_cast<uint2*>(g.dhu + o) = pack4(du[0], du[1], du[2], du[3]);
                *reinterpret_cast<uint2*>(g.act + o) = pack4(av[0], av[1], av[2], av[3]);
              }
            }
          });
        });
      }
    }
  });
}

// Per-expert row-tile prefix (mt_start) and experts ordered by row count,
// descending, ties by index (lpt).  One workgroup, E_loc <= 1024.
__global__ __launch_bounds__(1024) void gemm_sched_kernel(const int32_t* __restrict__ offsets,
                                                          int E_loc, int32_t* __restrict__ mt_start,
                                                          int32_t* __restrict__ lpt) {
  __shared__ int cnt[1024];
  __shared__ int wsum[16];
  const int e = threadIdx.x;
  const int n = (e < E_loc) ? offsets[e + 1] - offsets[e] : 0;
  cnt[e] = n;
  const int mt = (n + BM - 1) / BM;
  const int lane = e & 63, w = e >> 6;
  int incl = mt;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int v = __shfl_up(incl, o, 64);
    if (lane >= o) incl += v;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int base = 0;
  for (int i = 0; i < w; ++i) base += wsum[i];
  if (e < E_loc) mt_start[e] = base + incl - mt;
  if (e == E_loc - 1) mt_start[E_loc] = base + incl;
  if (e < E_loc) {
    int rank = 0;
    for (int o = 0; o < E_loc; ++o) {
      const int c = cnt[o];
      rank += (c > n) || (c == n && o < e);
    }
    lpt[rank] = e;
  }
}

struct GemmWs {
  int32_t* mt_start;
  int32_t* lpt;
  uint16_t* act;
  uint16_t* dhg;
  uint16_t* dhu;
};

GemmWs carve(void* ws, int64_t cap, int E_loc, int f, bool bwd) {
  char* p = static_cast<char*>(ws);
  GemmWs w{};
  w.mt_start = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (E_loc + 1), 256);
  w.lpt = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * E_loc, 256);
  const size_t act_bytes = align_up(sizeof(uint16_t) * static_cast<size_t>(cap) * f, 256);
  w.act = reinterpret_cast<uint16_t*>(p);
  p += act_bytes;
  if (bwd) {
    w.dhg = reinterpret_cast<uint16_t*>(p);
    p += act_bytes;
    w.dhu = reinterpret_cast<uint16_t*>(p);
  }
  return w;
}

template <int MODE>
hipError_t run_gemm(const GemmArgs& a, int64_t blocks, int kid, hipStream_t s) {
  if (blocks <= 0) return hipSuccess;
  prof_begin(kid, s);
  grouped_gemm_kernel<MODE><<<static_cast<unsigned>(blocks), 256, 0, s>>>(a);
  prof_end(kid, s);
  return hipGetLastError();
}

// Upper bound of the row tiles of all experts, rounded to a multiple of the
// XCD count (every logical tile must have a workgroup).
int64_t mgrid(int64_t cap, int E_loc, int NT) {
  const int64_t tiles = (ceil_div(cap, BM) + E_loc) * NT;
  return ceil_div(tiles, NXCD) * NXCD;
}

hipError_t sched(const int32_t* offsets, int E_loc, const GemmWs& w, hipStream_t s) {
  prof_begin(K_GEMM_SCHED, s);
  gemm_sched_kernel<<<1, 1024, 0, s>>>(offsets, E_loc, w.mt_start, w.lpt);
  prof_end(K_GEMM_SCHED, s);
  return hipGetLastError();
}

}  // namespace

size_t gemm_ws_bytes(int64_t cap, int E_loc, int d, int f, unsigned flags) {
  (void)d;
  const bool bwd = flags != 0;
  const size_t act_bytes = align_up(sizeof(uint16_t) * static_cast<size_t>(cap) * f, 256);
  return align_up(sizeof(int32_t) * (E_loc + 1), 256) + align_up(sizeof(int32_t) * E_loc, 256) +
         act_bytes * (bwd ? 3 : 1) + 256;
}

hipError_t launch_ffn_fwd(const uint16_t* x_perm, const int32_t* offsets, int E_loc, int64_t cap,
                          int d, int f, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, uint16_t* hg, uint16_t* hu, uint16_t* y,
                          void* ws, hipStream_t s) {
  GemmWs w = carve(ws, cap, E_loc, f, false);
  if (hipError_t e = sched(offsets, E_loc, w, s); e != hipSuccess) return e;
  GemmArgs a{};
  a.x_perm = x_perm; a.wg = wg; a.wu = wu; a.wd = wd;
  a.offsets = offsets; a.mt_start = w.mt_start; a.lpt = w.lpt;
  a.hg = hg; a.hu = hu; a.act = w.act; a.act_in = w.act; a.y = y;
  a.E_loc = E_loc; a.d = d; a.f = f;
  a.NT = static_cast<int>(ceil_div(f, BN / 2));
  if (hipError_t e = run_gemm<FWD_GATE_UP>(a, mgrid(cap, E_loc, a.NT), K_GEMM_FWD_GATE_UP, s);
      e != hipSuccess)
    return e;
  a.NT = static_cast<int>(ceil_div(d, BN));
  return run_gemm<FWD_DOWN>(a, mgrid(cap, E_loc, a.NT), K_GEMM_FWD_DOWN, s);
}

hipError_t launch_ffn_bwd(const uint16_t* dy, const uint16_t* x_perm, const uint16_t* hg,
                          const uint16_t* hu, const int32_t* offsets, int E_loc, int64_t cap,
                          int d, int f, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, uint16_t* dx, uint16_t* dwg, uint16_t* dwu,
                          uint16_t* dwd, unsigned flags, void* ws, hipStream_t s) {
  GemmWs w = carve(ws, cap, E_loc, f, true);
  if (hipError_t e = sched(offsets, E_loc, w, s); e != hipSuccess) return e;
  GemmArgs a{};
  a.x_perm = x_perm; a.wg = wg; a.wu = wu; a.wd = wd;
  a.hg_in = hg; a.hu_in = hu; a.dy = dy;
  a.offsets = offsets; a.mt_start = w.mt_start; a.lpt = w.lpt;
  a.dhg = w.dhg; a.dhu = w.dhu; a.act = w.act;
  a.dhg_in = w.dhg; a.dhu_in = w.dhu; a.act_in = w.act;
  a.dx = dx; a.dwg = dwg; a.dwu = dwu; a.dwd = dwd;
  a.E_loc = E_loc; a.d = d; a.f = f;
  a.NT = static_cast<int>(ceil_div(f, BN));
  if (hipError_t e = run_gemm<DGRAD_DOWN>(a, mgrid(cap, E_loc, a.NT), K_GEMM_DGRAD_DOWN, s);
      e != hipSuccess)
    return e;
  if (flags & MOE_BWD_DGRAD) {
    a.NT = static_cast<int>(ceil_div(d, BN));
    if (hipError_t e =
            run_gemm<DGRAD_GATE_UP>(a, mgrid(cap, E_loc, a.NT), K_GEMM_DGRAD_GATE_UP, s);
        e != hipSuccess)
      return e;
  }
  if (flags & MOE_BWD_WGRAD) {
    const int64_t egroups = ceil_div(E_loc, NXCD) * NXCD;
    a.MT = static_cast<int>(ceil_div(d, BM));
    a.NT = static_cast<int>(ceil_div(f, BN / 2));
    if (hipError_t e = run_gemm<WGRAD_GATE_UP>(a, egroups * a.MT * a.NT, K_GEMM_WGRAD_GATE_UP, s);
        e != hipSuccess)
      return e;
    a.MT = static_cast<int>(ceil_div(f, BM));
    a.NT = static_cast<int>(ceil_div(d, BN));
    if (hipError_t e = run_gemm<WGRAD_DOWN>(a, egroups * a.MT * a.NT, K_GEMM_WGRAD_DOWN, s);
        e != hipSuccess)
      return e;
  }
  return hipSuccess;
}

}  // namespace moe
