// Grouped SwiGLU expert GEMMs on gfx950 (bf16 MFMA, fp32 accumulation).
//
// Every GEMM of the expert FFN (forward gate/up and down, data gradients,
// weight gradients) is one instance of a single macro-tile kernel:
//   * 256 threads = 4 waves in a 2 x 2 grid; the block computes a 256 x 256
//     tile of C^T (rows = output columns n, cols = output rows m) with
//     v_mfma_f32_32x32x16_bf16, so each lane ends up holding four consecutive
//     output columns and stores 8 bytes at a time.
//   * Operands move global -> LDS with buffer_load_dwordx4 ... lds (no
//     register staging).  The buffer descriptor's range check turns every
//     tail (rows past an expert's segment, k past K, columns past N) into
//     zeros, so there is no padding and no per-element branching.
//   * K steps of 32 in a ring of 4 LDS stages (128 KiB of the 160 KiB):
//     loads run three steps ahead of the MFMAs; one barrier per step.
//   * Operands stored K-contiguous (activations in the forward pass and the
//     data gradients, weights in the data gradients) sit in LDS as
//     [256 rows][32 k] and feed the MFMA with ds_read_b128.  Operands stored
//     with the output index contiguous (weights in the forward pass,
//     everything in the weight gradients) keep that layout in LDS
//     ([32 k][128 cols] sub-tiles) and are read with ds_read_b64_tr_b16,
//     which transposes 4 x 16 blocks across each group of 16 lanes.
//     Both layouts carry a 16-byte-chunk XOR swizzle that makes the
//     fragment reads conflict-free.
//   * Variable-size expert segments: a tiny scheduler kernel turns
//     expert_offsets into per-expert tile counts on the device (no host
//     synchronisation, no padding to a capacity).  An expert without rows
//     gets no forward tiles and zero weight gradients.
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
constexpr int BK = 32;       // k per pipeline stage
constexpr int NST = 4;       // LDS stages
constexpr int OP_BYTES = 256 * BK * 2;     // one operand tile per stage (16 KiB)
constexpr int STAGE_BYTES = 2 * OP_BYTES;  // A + B (32 KiB)
constexpr int LOADS = 4;     // 16-byte direct loads per lane, per operand and stage
constexpr int NXCD = 8;
constexpr uint32_t OOB = 0x80000000u;  // buffer offset past every range: reads as zero

enum Mode {
  FWD_GATE_UP = 0,  // Hg, Hu, A  = X Wg, X Wu, silu(Hg) Hu       (dual B, K = d)
  FWD_DOWN,         // Y = A Wd                                    (K = f)
  DGRAD_DOWN,       // dA = dY Wd^T -> dHg, dHu, A                 (K = d)
  DGRAD_GATE_UP,    // dX = dHg Wg^T + dHu Wu^T                    (K = 2f)
  WGRAD_GATE_UP,    // dWg, dWu = X^T dHg, X^T dHu                 (dual B, K = n_e)
  WGRAD_DOWN        // dWd = A^T dY                                (K = n_e)
};

typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;

// Buffer descriptor (gfx9 layout): base, no stride, `bytes` of range
// (clamped to [0, 2^31 - 16]; a negative range means nothing is readable).
__device__ __forceinline__ i32x4 make_rsrc(const void* p, int64_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(p);
  i32x4 r;
  r[0] = static_cast<int>(a & 0xffffffffu);
  r[1] = static_cast<int>((a >> 32) & 0xffffu);
  r[2] = static_cast<int>(bytes <= 0 ? 0 : (bytes > 0x7ffffff0 ? 0x7ffffff0 : bytes));
  r[3] = 0x00020000;
  r[0] = __builtin_amdgcn_readfirstlane(r[0]);
  r[1] = __builtin_amdgcn_readfirstlane(r[1]);
  r[2] = __builtin_amdgcn_readfirstlane(r[2]);
  r[3] = __builtin_amdgcn_readfirstlane(r[3]);
  return r;
}

#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
// 16 bytes per lane, global -> LDS; lane i writes LDS [lds + 16 i, +16).
// Issued as inline asm so the compiler does not wait for it at every
// barrier; completion is tracked by hand with vmcnt.
__device__ __forceinline__ void load_lds16(const i32x4& rsrc, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(lds), "v"(voff), "s"(rsrc)
               : "memory", "m0");
}
#pragma clang diagnostic pop

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

// ------------------------------------------------------- K-major operand
// Tile rows r (m or n) with k contiguous: element (r, k) of source s at
// byte r*ld + 2k from its base.  Dual-K: steps [0, nk0) read source 0,
// steps [nk0, nk) source 1 (k restarts at 0).  LDS: [256][32] bf16,
// 64-byte rows, chunk c of row r at ((c ^ ((r >> 1) & 3)) << 4).
__device__ __forceinline__ int koff(int r, int c) { return r * (BK * 2) + ((c ^ ((r >> 1) & 3)) << 4); }

struct KOperand {
  i32x4 rsrc0, rsrc1;
  uint32_t ld;      // row pitch in bytes
  int rows;         // valid tile rows
  int kmax0, kmax1; // valid k of source 0 / 1
  int nk0;          // steps of source 0

  // Per load q (0..3) of this wave, lane l covers tile row
  // r = 16 (4 wave + q) + l / 4 and 16-byte chunk lc = (l % 4) ^ ((r / 2) % 4).
  __device__ __forceinline__ void issue(int kt, uint32_t lds_op, int wave, int lane) const {
    const bool s1 = kt >= nk0;
    const int k0 = (s1 ? kt - nk0 : kt) * BK;
    const int km = s1 ? kmax1 : kmax0;
    const i32x4 rs = s1 ? rsrc1 : rsrc0;
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int r = (wave * LOADS + q) * 16 + (lane >> 2);
      const int lc = (lane & 3) ^ ((r >> 1) & 3);
      const bool ok = r < rows && k0 + lc * 8 < km;
      const uint32_t v = static_cast<uint32_t>(r) * ld + static_cast<uint32_t>(lc * 16 + k0 * 2);
      load_lds16(rs, ok ? v : OOB, lds_op + (wave * LOADS + q) * 1024);
    }
  }
  // MFMA fragment: 8 consecutive k (k-group `kg` of substep s) of tile row r
  static __device__ __forceinline__ bf16x8 frag(const lds_char* t, int r, int s, int kg) {
    return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(t + koff(r, 2 * s + kg));
  }
};

// ------------------------------------------------------- N-major operand
// Stored [k][cols] with the tile index contiguous: element (k, c) at byte
// k*ld + 2c of the sub-tile's base.  The tile's 256 columns are two
// sub-tiles of 128 (sub-tile j starts at ptr_j, has cols_j valid columns and
// range_j readable bytes); k < kmax valid.  The descriptor base advances
// with the K step, so lane offsets stay below 32 rows.  LDS: per sub-tile
// [32][128] bf16, 256-byte rows, chunk c of row k at ((c ^ (2 (k & 3))) << 4).
__device__ __forceinline__ int noff(int k, int col) {
  return k * 256 + ((((col >> 3) ^ (2 * (k & 3)))) << 4) + ((col >> 2) & 1) * 8;
}

struct NOperand {
  const uint16_t* ptr0;
  const uint16_t* ptr1;
  int64_t range0, range1;
  uint32_t ld;
  int cols0, cols1;
  int kmax;

  // Per load q (0..3) of this wave: instruction I = 4 wave + q covers rows
  // 4 (I % 8) .. +3 of sub-tile I / 8; lane l takes row k = 4 (I % 8) + l / 16
  // and column 8 ((l % 16) ^ (2 (k % 4))).
  __device__ __forceinline__ void issue(int kt, uint32_t lds_op, int wave, int lane) const {
    const int k0 = kt * BK;
    const int64_t adv = static_cast<int64_t>(k0) * ld;
    const i32x4 r0 = make_rsrc(reinterpret_cast<const char*>(ptr0) + adv, range0 - adv);
    const i32x4 r1 = make_rsrc(reinterpret_cast<const char*>(ptr1) + adv, range1 - adv);
#pragma unroll
    for (int q = 0; q < LOADS; ++q) {
      const int I = wave * LOADS + q;
      const int k = (I & 7) * 4 + (lane >> 4);
      const int col = ((lane & 15) ^ (2 * (k & 3))) * 8;
      const bool ok = col < ((I >> 3) ? cols1 : cols0) && k0 + k < kmax;
      const uint32_t v = static_cast<uint32_t>(k) * ld + static_cast<uint32_t>(col) * 2u;
      load_lds16((I >> 3) ? r1 : r0, ok ? v : OOB,
                 lds_op + (I >> 3) * (OP_BYTES / 2) + (I & 7) * 1024);
    }
  }
  // MFMA fragment of tile column block c0 (multiple of 32): lane l gets
  // 8 consecutive k (k-group l/32 of substep s) of column c0 + l%32, built
  // from two transposing reads of 4 k each.
  static __device__ __forceinline__ bf16x8 frag(const lds_char* t, int c0, int s, int lane) {
    const int g = lane >> 4, r = lane & 15;
    const int st = c0 >> 7;
    const int col = (c0 & 127) + 16 * (g & 1) + 4 * (r & 3);
    const int k = 16 * s + 8 * (g >> 1) + (r >> 2);
    const lds_char* b = t + st * (OP_BYTES / 2);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(b + noff(k, col)));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(b + noff(k + 4, col)));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
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


// One output tile of one expert.
struct Tile {
  bool valid;
  int e, m0, n0, seg, ne, nk;
};

// The sequence of tiles one workgroup computes.  The grid has one workgroup
// per CU; workgroup b runs on XCD b % 8 as CU slot b / 8 of that XCD.
//  * Row-grouped GEMMs: logical tiles (expert-major; inside an expert the
//    row tiles of one column tile are adjacent) are cut into 8 equal
//    contiguous ranges, one per XCD, dealt round-robin to the XCD's CUs.
//  * Weight gradients: groups (expert, row tile) in LPT order (experts by
//    rows, descending) are dealt to XCDs in snake order (0..7, 7..0, ...),
//    which balances skewed loads and spreads a large expert over all XCDs;
//    the column tiles of a group are adjacent on its XCD.
// Schedule tables of one launch, copied to LDS at kernel start: tile
// decoding then never waits on the vector-memory counter, which the
// in-flight operand loads use.
struct Tables {
  const int* mt_start;  // [E_loc + 1]
  const int* offsets;   // [E_loc + 1]
  const int* lpt;       // [E_loc]
};

template <int MODE>
struct TileIter {
  static constexpr bool WG = (MODE == WGRAD_GATE_UP || MODE == WGRAD_DOWN);
  static constexpr bool DUAL = (MODE == FWD_GATE_UP || MODE == WGRAD_GATE_UP);
  int xcd, j, cpx, i;
  int total, end;  // row-grouped: tile count, end of this XCD's range
  int gq, lim;     // weight gradients: group count, XCD-local tile bound
  bool zeros;      // weight gradients: visit only the tiles of experts without rows

  __device__ __forceinline__ void init(const GemmArgs& g, const Tables& tb, bool zero_tiles = false) {
    zeros = zero_tiles;
    cpx = gridDim.x / NXCD;
    xcd = blockIdx.x % NXCD;
    j = blockIdx.x / NXCD;
    i = 0;
    if constexpr (!WG) {
      total = tb.mt_start[g.E_loc] * g.NT;
      const int per = (total + NXCD - 1) / NXCD;
      end = min((xcd + 1) * per, total);
      total = xcd * per;  // start of this XCD's range
    } else {
      gq = g.E_loc * g.MT;
      lim = 2 * ((gq + 15) / 16) * g.NT;
    }
  }
  __device__ __forceinline__ Tile next(const GemmArgs& g, const Tables& tb) {
    Tile t;
    t.valid = false;
    if constexpr (!WG) {
      const int L = total + j + cpx * i;
      ++i;
      if (L >= end) return t;
      int lo = 0, hi = g.E_loc;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (tb.mt_start[mid] * g.NT <= L) lo = mid; else hi = mid;
      }
      t.e = __builtin_amdgcn_readfirstlane(lo);
      const int ms0 = __builtin_amdgcn_readfirstlane(tb.mt_start[lo]);
      const int mt_e = __builtin_amdgcn_readfirstlane(tb.mt_start[lo + 1]) - ms0;
      const int local = L - ms0 * g.NT;
      t.m0 = (local % mt_e) * BM;
      t.n0 = (local / mt_e) * (DUAL ? BN / 2 : BN);
      t.seg = __builtin_amdgcn_readfirstlane(tb.offsets[lo]);
      t.ne = __builtin_amdgcn_readfirstlane(tb.offsets[lo + 1]) - t.seg;
      const int K = (MODE == FWD_GATE_UP || MODE == DGRAD_DOWN) ? g.d : g.f;
      t.nk = ((K + BK - 1) / BK) * (MODE == DGRAD_GATE_UP ? 2 : 1);
      t.valid = true;
      return t;
    } else {
      while (true) {
        const int lt = j + cpx * i;
        ++i;
        if (lt >= lim) return t;
        const int k = lt / g.NT, nt = lt % g.NT;
        const int q = 16 * (k >> 1) + ((k & 1) ? 15 - xcd : xcd);
        if (q >= gq) continue;
        t.e = __builtin_amdgcn_readfirstlane(tb.lpt[q / g.MT]);
        t.m0 = (q % g.MT) * BM;
        t.n0 = nt * (DUAL ? BN / 2 : BN);
        t.seg = __builtin_amdgcn_readfirstlane(tb.offsets[t.e]);
        t.ne = __builtin_amdgcn_readfirstlane(tb.offsets[t.e + 1]) - t.seg;
        t.nk = (t.ne + BK - 1) / BK;
        if (t.nk == 0 && !zeros) continue;
        if (t.nk != 0 && zeros) continue;
        t.valid = true;
        return t;
      }
    }
  }
};

template <int MODE>
__global__ __launch_bounds__(256, 1) void grouped_gemm_kernel(GemmArgs g) {
  __shared__ __align__(1024) char lds[NST * STAGE_BYTES];
  __shared__ int tab[3 * MOE_MAX_E + 2];
  constexpr bool WGRAD = (MODE == WGRAD_GATE_UP || MODE == WGRAD_DOWN);
  constexpr bool DUAL = (MODE == FWD_GATE_UP || MODE == WGRAD_GATE_UP);
  constexpr bool A_N = WGRAD;                                        // A side N-major?
  constexpr bool B_K = (MODE == DGRAD_DOWN || MODE == DGRAD_GATE_UP);  // B side K-major?
  using AOp = typename std::conditional<A_N, NOperand, KOperand>::type;
  using BOp = typename std::conditional<B_K, KOperand, NOperand>::type;

  const int d = g.d, f = g.f;
  const int64_t wdf = static_cast<int64_t>(d) * f;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w >> 1, wn = w & 1;
  const int l32 = lane & 31, lh = lane >> 5;

  // ------------------------------------------------------- operand setup
  // A side = rows m of the output, B side = columns n of the output.
  auto setup = [&](const Tile& tl, AOp& A, BOp& B) __attribute__((always_inline)) {
    const int e = tl.e, m0 = tl.m0, n0 = tl.n0, seg = tl.seg, ne = tl.ne;
    if constexpr (MODE == FWD_GATE_UP) {
      const uint16_t* xa = g.x_perm + (int64_t)(seg + m0) * d;
      A.rsrc0 = A.rsrc1 = make_rsrc(xa, (int64_t)(ne - m0) * d * 2);
      A.ld = d * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = d; A.nk0 = (d + BK - 1) / BK;
      B.ptr0 = g.wg + e * wdf + n0; B.range0 = (wdf - n0) * 2;
      B.ptr1 = g.wu + e * wdf + n0; B.range1 = (wdf - n0) * 2;
      B.ld = f * 2; B.cols0 = B.cols1 = f - n0; B.kmax = d;
    } else if constexpr (MODE == FWD_DOWN) {
      const uint16_t* aa = g.act_in + (int64_t)(seg + m0) * f;
      A.rsrc0 = A.rsrc1 = make_rsrc(aa, (int64_t)(ne - m0) * f * 2);
      A.ld = f * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = f; A.nk0 = (f + BK - 1) / BK;
      B.ptr0 = g.wd + e * wdf + n0; B.range0 = (wdf - n0) * 2;
      B.ptr1 = B.ptr0 + 128; B.range1 = (wdf - n0 - 128) * 2;
      B.ld = d * 2; B.cols0 = d - n0; B.cols1 = d - n0 - 128; B.kmax = f;
    } else if constexpr (MODE == DGRAD_DOWN) {
      const uint16_t* ya = g.dy + (int64_t)(seg + m0) * d;
      A.rsrc0 = A.rsrc1 = make_rsrc(ya, (int64_t)(ne - m0) * d * 2);
      A.ld = d * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = d; A.nk0 = (d + BK - 1) / BK;
      const uint16_t* wb = g.wd + e * wdf + (int64_t)n0 * d;
      B.rsrc0 = B.rsrc1 = make_rsrc(wb, (int64_t)(f - n0) * d * 2);
      B.ld = d * 2; B.rows = f - n0; B.kmax0 = B.kmax1 = d; B.nk0 = A.nk0;
    } else if constexpr (MODE == DGRAD_GATE_UP) {
      const int64_t ro = (int64_t)(seg + m0) * f;
      A.rsrc0 = make_rsrc(g.dhg_in + ro, (int64_t)(ne - m0) * f * 2);
      A.rsrc1 = make_rsrc(g.dhu_in + ro, (int64_t)(ne - m0) * f * 2);
      A.ld = f * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = f; A.nk0 = (f + BK - 1) / BK;
      const int64_t wo = e * wdf + (int64_t)n0 * f;
      B.rsrc0 = make_rsrc(g.wg + wo, (int64_t)(d - n0) * f * 2);
      B.rsrc1 = make_rsrc(g.wu + wo, (int64_t)(d - n0) * f * 2);
      B.ld = f * 2; B.rows = d - n0; B.kmax0 = B.kmax1 = f; B.nk0 = A.nk0;
    } else if constexpr (MODE == WGRAD_GATE_UP) {
      A.ptr0 = g.x_perm + (int64_t)seg * d + m0; A.range0 = ((int64_t)ne * d - m0) * 2;
      A.ptr1 = A.ptr0 + 128; A.range1 = A.range0 - 256;
      A.ld = d * 2; A.cols0 = d - m0; A.cols1 = d - m0 - 128; A.kmax = ne;
      B.ptr0 = g.dhg_in + (int64_t)seg * f + n0; B.range0 = ((int64_t)ne * f - n0) * 2;
      B.ptr1 = g.dhu_in + (int64_t)seg * f + n0; B.range1 = B.range0;
      B.ld = f * 2; B.cols0 = B.cols1 = f - n0; B.kmax = ne;
    } else {  // WGRAD_DOWN
      A.ptr0 = g.act_in + (int64_t)seg * f + m0; A.range0 = ((int64_t)ne * f - m0) * 2;
      A.ptr1 = A.ptr0 + 128; A.range1 = A.range0 - 256;
      A.ld = f * 2; A.cols0 = f - m0; A.cols1 = f - m0 - 128; A.kmax = ne;
      B.ptr0 = g.dy + (int64_t)seg * d + n0; B.range0 = ((int64_t)ne * d - n0) * 2;
      B.ptr1 = B.ptr0 + 128; B.range1 = B.range0 - 256;
      B.ld = d * 2; B.cols0 = d - n0; B.cols1 = d - n0 - 128; B.kmax = ne;
    }
  };

  int arow[4], brow[4];  // first tile row of each 32-row MFMA block
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    arow[i] = wm * 128 + 32 * i;
    if constexpr (DUAL)
      brow[i] = (i < 2 ? 0 : BN / 2) + wn * 64 + 32 * (i & 1);
    else
      brow[i] = wn * 128 + 32 * i;
  }

  f32x16 acc[4][4];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][jj][r] = 0.0f;
  };

  // ------------------------------------------------------------ epilogue
  // acc[i][j][4q + u]: output row m = arow[i] + l32 (tile-relative),
  // output column n = brow[j] + 8q + 4*lh + u.
  auto epilogue = [&](const Tile& tl) __attribute__((always_inline)) {
    const int e = tl.e, m0 = tl.m0, n0 = tl.n0, seg = tl.seg, ne = tl.ne;
    int arow[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) arow[i] = wm * 128 + 32 * i + l32;
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
  };


  // zero weight-gradient tile (expert without rows)
  auto zero_tile = [&](const Tile& tl) __attribute__((always_inline)) {
    const int R = (MODE == WGRAD_GATE_UP) ? d : f;   // output rows
    const int C = (MODE == WGRAD_GATE_UP) ? f : d;   // output columns
    const int cw = DUAL ? BN / 2 : BN;               // tile columns per output
    const int nout = DUAL ? 2 : 1;
    for (int idx = threadIdx.x; idx < BM * (cw / 8) * nout; idx += 256) {
      const int o = idx / (BM * (cw / 8));
      const int rem = idx % (BM * (cw / 8));
      const int r = tl.m0 + rem / (cw / 8), c = tl.n0 + (rem % (cw / 8)) * 8;
      if (r < R && c < C) {
        uint16_t* base = (MODE == WGRAD_GATE_UP) ? (o ? g.dwu : g.dwg) : g.dwd;
        *reinterpret_cast<uint4*>(base + tl.e * wdf + (int64_t)r * C + c) = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };

  const lds_char* ldsp = (const lds_char*)(lds);  // address-space cast
  const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ldsp));
  struct Frags {
    bf16x8 a[4], b[4];
  };
  // fragments of half step `s` (16 k) of LDS stage `stage`
  auto load_frags = [&](Frags& F, int stage, int s) __attribute__((always_inline)) {
    const lds_char* ta = ldsp + stage * STAGE_BYTES;
    const lds_char* tb = ta + OP_BYTES;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (A_N) F.a[i] = AOp::frag(ta, arow[i], s, lane);
      else F.a[i] = AOp::frag(ta, arow[i] + l32, s, lh);
    }
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      if constexpr (B_K) F.b[jj] = BOp::frag(tb, brow[jj] + l32, s, lh);
      else F.b[jj] = BOp::frag(tb, brow[jj], s, lane);
    }
  };
  auto mma = [&](const Frags& F) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 4; ++jj)
        acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.b[jj], F.a[i], acc[i][jj], 0, 0, 0);
  };
  auto wait_stages = [&](int n) __attribute__((always_inline)) {  // at most n stages of this wave's loads in flight
    if (n >= 3) wait_vmcnt<6 * LOADS>();
    else if (n == 2) wait_vmcnt<4 * LOADS>();
    else if (n == 1) wait_vmcnt<2 * LOADS>();
    else wait_vmcnt<0>();
  };

  // ---------------------------------------------------------- tile stream
  // The workgroup's tiles form one stream of K steps.  Loads run up to
  // NST steps ahead in a ring of NST LDS stages, across tile boundaries, so
  // the next tile's first steps are in flight while the current tile
  // finishes and writes its epilogue.  Each step is two half steps of 16 k:
  // the fragments of the next half step are read while the MFMAs of the
  // current one run, and the step's one barrier sits between its halves.
  for (int i = threadIdx.x; i <= g.E_loc; i += 256) {
    tab[i] = g.mt_start[i];
    tab[MOE_MAX_E + 1 + i] = g.offsets[i];
    if (i < g.E_loc) tab[2 * MOE_MAX_E + 2 + i] = g.lpt[i];
  }
  __syncthreads();
  const Tables tb{tab, tab + MOE_MAX_E + 1, tab + 2 * MOE_MAX_E + 2};
  TileIter<MODE> itc, iti;
  itc.init(g, tb);
  iti.init(g, tb);
  zero_acc();
  Tile tc = itc.next(g, tb);
  Tile ti = iti.next(g, tb);
  if (tc.valid) {
    AOp A;  // operands of the tile being loaded
    BOp B;
    bool have = false;
    int kti = 0, nIssued = 0;
    auto issue_one = [&]() __attribute__((always_inline)) {
      if (ti.valid && kti >= ti.nk) {
        ti = iti.next(g, tb);
        kti = 0;
        have = false;
      }
      if (!ti.valid) return;
      if (!have) {
        setup(ti, A, B);
        have = true;
      }
      const uint32_t st = lds0 + (nIssued % NST) * STAGE_BYTES;
      A.issue(kti, st, w, lane);
      B.issue(kti, st + OP_BYTES, w, lane);
      ++kti;
      ++nIssued;
    };
#pragma unroll
    for (int p = 0; p < NST; ++p) issue_one();

    Frags cur, nxt;
    wait_stages(nIssued - 1);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    load_frags(cur, 0, 0);
    int s = 0;  // step of the stream being computed
    bool after_epi = false;
    // step s + 1 has landed in LDS and stage s may be refilled (barrier),
    // then the load stream advances by one step
    auto sync_and_issue = [&]() __attribute__((always_inline)) {
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave is done with stage s
      if (after_epi) {
        wait_vmcnt<0>();  // epilogue stores share the counter
      } else {
        const int later = nIssued - s - 2;  // steps issued after s + 1
        wait_stages(later < 2 ? later : 2);
      }
      after_epi = false;
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);
      issue_one();  // into stage s % NST
    };
    while (true) {
      for (int kk = 0; kk + 1 < tc.nk; ++kk) {  // all steps of the tile but its last
        load_frags(nxt, s % NST, 1);
        __builtin_amdgcn_sched_barrier(0);
        mma(cur);
        __builtin_amdgcn_sched_barrier(0);
        sync_and_issue();  // step s + 1 exists: it is this tile's
        load_frags(cur, (s + 1) % NST, 0);
        __builtin_amdgcn_sched_barrier(0);
        mma(nxt);
        __builtin_amdgcn_sched_barrier(0);
        ++s;
      }
      // last step of the tile
      load_frags(nxt, s % NST, 1);
      __builtin_amdgcn_sched_barrier(0);
      mma(cur);
      __builtin_amdgcn_sched_barrier(0);
      const bool more = nIssued > s + 1;
      if (more) sync_and_issue();
      mma(nxt);
      __builtin_amdgcn_sched_barrier(0);
      ++s;
      epilogue(tc);
      zero_acc();
      after_epi = true;
      if (!more) break;
      tc = itc.next(g, tb);
      load_frags(cur, s % NST, 0);  // first half of the next tile's first step
    }
  }
  if constexpr (WGRAD) {
    // experts without rows: their weight gradients are exact zeros
    TileIter<MODE> itz;
    itz.init(g, tb, true);
    for (Tile tz = itz.next(g, tb); tz.valid; tz = itz.next(g, tb)) zero_tile(tz);
  }
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

// Persistent grid: one workgroup per CU (a multiple of the 8 XCDs).
int64_t pgrid() {
  static int cus = [] {
    int dev = 0, n = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
      n = 256;
    return n;
  }();
  const int64_t g = (cus / NXCD) * NXCD;
  return g > 0 ? g : NXCD;
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
  if (hipError_t e = run_gemm<FWD_GATE_UP>(a, pgrid(), K_GEMM_FWD_GATE_UP, s);
      e != hipSuccess)
    return e;
  a.NT = static_cast<int>(ceil_div(d, BN));
  return run_gemm<FWD_DOWN>(a, pgrid(), K_GEMM_FWD_DOWN, s);
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
  if (hipError_t e = run_gemm<DGRAD_DOWN>(a, pgrid(), K_GEMM_DGRAD_DOWN, s);
      e != hipSuccess)
    return e;
  if (flags & MOE_BWD_DGRAD) {
    a.NT = static_cast<int>(ceil_div(d, BN));
    if (hipError_t e =
            run_gemm<DGRAD_GATE_UP>(a, pgrid(), K_GEMM_DGRAD_GATE_UP, s);
        e != hipSuccess)
      return e;
  }
  if (flags & MOE_BWD_WGRAD) {
    a.MT = static_cast<int>(ceil_div(d, BM));
    a.NT = static_cast<int>(ceil_div(f, BN / 2));
    if (hipError_t e = run_gemm<WGRAD_GATE_UP>(a, pgrid(), K_GEMM_WGRAD_GATE_UP, s);
        e != hipSuccess)
      return e;
    a.MT = static_cast<int>(ceil_div(f, BM));
    a.NT = static_cast<int>(ceil_div(d, BN));
    if (hipError_t e = run_gemm<WGRAD_DOWN>(a, pgrid(), K_GEMM_WGRAD_DOWN, s);
        e != hipSuccess)
      return e;
  }
  return hipSuccess;
}

}  // namespace moe
