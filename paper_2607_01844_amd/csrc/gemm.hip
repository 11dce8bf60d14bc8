// Grouped SwiGLU expert GEMMs on gfx950 (bf16 MFMA, fp32 accumulation).
//
// Every GEMM of the expert FFN (forward gate/up and down, data gradients,
// weight gradients) is one instance of a single macro-tile kernel:
//   * 512 threads = 8 waves (two per SIMD) in a 2 x 4 grid; the block
//     computes a 256 x 256 tile of C^T (rows = output columns n, cols =
//     output rows m) with v_mfma_f32_32x32x16_bf16, each wave 128 rows x 64
//     columns; the epilogue passes each wave's block through LDS so that
//     every global store moves 16 bytes per lane.
//   * Operands move global -> LDS with buffer_load_dwordx4 ... lds (no
//     register staging).  Out-of-range lanes (rows past an expert's segment,
//     k past K, columns past N) get an offset past the buffer descriptor's
//     range and read zeros, so there is no padding and no per-element
//     branching.
//   * K steps of 64 through a ring of five 32 KiB LDS slots (all 160 KiB):
//     two for operand A (loaded one step ahead) and three for operand B (two
//     steps ahead); one barrier per step.  Each operand's loads of a tile
//     are prepared once when the tile starts (descriptors in scalar
//     registers, lane offsets in vector registers), so a step's loads cost
//     little more than the loads themselves; they go out between the MFMAs
//     that follow the barrier, and the next sub-step's fragment reads go out
//     one by one between the current sub-step's MFMAs.  Near a tile's end the
//     look-ahead loads fetch the next tile's first steps.  A step of 64 k
//     makes every row of a K-contiguous tile one full 128-byte line, which
//     the memory path moves at twice the rate of 64-byte halves.
//   * The weight gradients (grouped, and the vocabulary's dW), which read
//     both operands with transposing LDS reads, run the same ring in a
//     ping-pong schedule when their tiles are long: the two waves of each
//     SIMD take turns, one running a half step of MFMAs while the other
//     reads its next fragments, with a barrier between turns.  One group of
//     four waves issues all operand loads and the other all output stores,
//     so no wave that waits for operands has stores ahead of them.
//   * Operands stored K-contiguous (activations in the forward pass and the
//     data gradients, weights in the data gradients) sit in LDS as
//     [256 rows][64 k] and feed the MFMA with ds_read_b128.  Operands stored
//     with the output index contiguous (weights in the forward pass,
//     everything in the weight gradients) keep that layout in LDS
//     ([64 k][128 cols] sub-tiles) and are read with ds_read_b64_tr_b16,
//     which transposes 4 x 16 blocks across each group of 16 lanes.
//     Both layouts carry a 16-byte-chunk XOR swizzle that makes the
//     fragment reads conflict-free.
//   * Variable-size expert segments: a tiny scheduler kernel turns
//     expert_offsets into per-expert tile counts on the device (no host
//     synchronisation, no padding to a capacity).  An expert without rows
//     gets no forward tiles and zero weight gradients.
//   * XCD-aware order: gfx950 hands consecutive workgroups to its 8 XCDs in
//     turn, and each XCD has its own L2.  Logical tiles are laid out so each
//     XCD runs a contiguous range of them, walked in groups of 4 or 8 row
//     tiles: the 32 tiles an XCD runs at a time form a 4 x 8 or 8 x 4 block
//     of one expert that shares its row and column slabs of the operands in
//     that L2.
//   * Dense modes run the same loop on plain products (the router's
//     backward and the blockwise vocabulary loss) with their own epilogues.
#include "common.h"

namespace moe {
namespace {

constexpr int BM = 256;      // tile rows on the operand-A side (m)
constexpr int BN = 256;      // tile rows on the operand-B side (n)
constexpr int BK = 64;       // k per step (128-byte rows of a K-contiguous tile)
constexpr int UNIT = 256 * BK * 2;  // one operand tile of one step in LDS (32 KiB)
constexpr int HALF = UNIT / 2;      // half a step (32 k) of an N-contiguous tile
constexpr int NWAVE = 8;     // waves per workgroup: two per SIMD
constexpr int NTHR = 64 * NWAVE;
constexpr int NRING = 5;     // LDS ring slots of UNIT bytes (160 KiB)
constexpr int PATCH_BYTES = UNIT / NWAVE;  // per-wave epilogue staging (4 KiB)
constexpr int NXCD = 8;
constexpr uint32_t OOB = 0x80000000u;  // buffer offset past every range: reads as zero

enum Mode {
  FWD_GATE_UP = 0,  // Hg, Hu, A  = X Wg, X Wu, silu(Hg) Hu       (dual B, K = d)
  FWD_DOWN,         // Y = A Wd                                    (K = f)
  DGRAD_DOWN,       // dA = dY Wd^T -> dHg, dHu, A                 (K = d)
  DGRAD_GATE_UP,    // dX = dHg Wg^T + dHu Wu^T                    (K = 2f)
  WGRAD_GATE_UP,    // dWg, dWu = X^T dHg, X^T dHu                 (dual B, K = n_e)
  WGRAD_DOWN,       // dWd = A^T dY                                (K = n_e)
  // Dense products: `batches` independent products of one shape, batch b
  // covering K rows [b kspan, min((b + 1) kspan, K)) of the contraction.
  RT_DW,            // router: part[b] = X_b^T (DLhi_b + DLlo_b), fp32   (dual B)
  RT_DX,            // router: dx = bf16([dx +] DL3 W3), K = 3E
  VOC_FWD,          // vocabulary: per row and 64 columns (max, sum exp), target logit
  VOC_GRAD,         // vocabulary: G = bf16(dl ([v == t] - exp(y - lse)))
  VOC_DX,           // vocabulary: dxa[b] (+)= G_b W_b^T, fp32
  VOC_DW            // vocabulary: dW[:, block] = X^T G, bf16
};

template <int MODE>
struct Traits {
  static constexpr bool DENSE = MODE >= RT_DW;
  // operand A stored with the output row index contiguous (read transposed)
  static constexpr bool A_N =
      MODE == WGRAD_GATE_UP || MODE == WGRAD_DOWN || MODE == RT_DW || MODE == VOC_DW;
  // operand B stored K-contiguous
  static constexpr bool B_K = MODE == DGRAD_DOWN || MODE == DGRAD_GATE_UP || MODE == VOC_DX;
  // B tile = 128 columns of each of two sources (same output column)
  static constexpr bool DUAL = MODE == FWD_GATE_UP || MODE == WGRAD_GATE_UP || MODE == RT_DW;
  // grouped weight gradients (K = an expert's rows, zero tiles for empty experts)
  static constexpr bool WG = MODE == WGRAD_GATE_UP || MODE == WGRAD_DOWN;
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
// The descriptor and LDS address are wave-uniform; readfirstlane states it
// so that they always reach the instruction in scalar registers.
__device__ __forceinline__ void load_lds16(const i32x4& rsrc, uint32_t voff, uint32_t lds) {
  i32x4 r;
  r[0] = __builtin_amdgcn_readfirstlane(rsrc[0]);
  r[1] = __builtin_amdgcn_readfirstlane(rsrc[1]);
  r[2] = __builtin_amdgcn_readfirstlane(rsrc[2]);
  r[3] = __builtin_amdgcn_readfirstlane(rsrc[3]);
  const uint32_t l = __builtin_amdgcn_readfirstlane(lds);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(l), "v"(voff), "s"(r)
               : "memory", "m0");
}
#pragma clang diagnostic pop

// A value the optimiser cannot see through: per-lane load offsets derived
// from it are recomputed at each issue instead of being hoisted out of the
// K loop, where they would be spilled and reloaded (and a scratch reload
// waits for every load in flight).
__device__ __forceinline__ int opaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}

// Compiler-visible s_waitcnt lgkmcnt(0) (vmcnt and expcnt left at their
// maximum): after code that may have issued scalar loads (kernel arguments,
// schedule tables), so that the waitcnt pass, which must assume such loads
// return out of order, does not turn the next fragment wait into a full one.
__device__ __forceinline__ void lgkm_drained() { __builtin_amdgcn_s_waitcnt(0xc07f); }

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory");
}

typedef uint32_t u32x4a __attribute__((ext_vector_type(4)));
// Eight 16-byte loads into registers (four from each of two buffers, same
// offsets) that complete inside the statement: the compiler never sees them
// in flight, so its own counter bookkeeping stays exact around the K loop.
// Waits for every vector-memory operation of the wave.
__device__ __forceinline__ void load_2x4_wait(const i32x4& ra, const i32x4& rb, const uint32_t (&off)[4],
                                              u32x4a (&a)[4], u32x4a (&b)[4]) {
  asm volatile(
      "buffer_load_dwordx4 %0, %8, %12, 0 offen\n\t"
      "buffer_load_dwordx4 %1, %9, %12, 0 offen\n\t"
      "buffer_load_dwordx4 %2, %10, %12, 0 offen\n\t"
      "buffer_load_dwordx4 %3, %11, %12, 0 offen\n\t"
      "buffer_load_dwordx4 %4, %8, %13, 0 offen\n\t"
      "buffer_load_dwordx4 %5, %9, %13, 0 offen\n\t"
      "buffer_load_dwordx4 %6, %10, %13, 0 offen\n\t"
      "buffer_load_dwordx4 %7, %11, %13, 0 offen\n\t"
      "s_waitcnt vmcnt(0)"
      : "=&v"(a[0]), "=&v"(a[1]), "=&v"(a[2]), "=&v"(a[3]), "=&v"(b[0]), "=&v"(b[1]), "=&v"(b[2]),
        "=&v"(b[3])
      : "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "s"(ra), "s"(rb)
      : "memory");
}
// ------------------------------------------------------- K-major operand
// Tile rows r (m or n) with k contiguous: element (r, k) of source s at
// byte r*ld + 2k from its base.  Dual-K: steps [0, nk0) read source 0,
// steps [nk0, nk) source 1 (k restarts at 0).  LDS: [256][64] bf16,
// 128-byte rows, 16-byte chunk c of row r at ((c ^ ((r / 2) % 8)) << 4): the
// 16 rows one ds_read_b128 pass covers (64 banks of 4 bytes) hit 16
// different 16-byte bank groups.
__device__ __forceinline__ int koff(int r, int c) { return r * (BK * 2) + ((c ^ ((r >> 1) & 7)) << 4); }

struct KOperand {
  i32x4 rsrc0, rsrc1;
  uint32_t ld;      // row pitch in bytes
  int rows;         // valid tile rows
  int kmax0, kmax1; // valid k of source 0 / 1
  int nk0;          // steps of source 0

  // MFMA fragment: 8 consecutive k (k-group `kg` of substep s) of tile row r
  static __device__ __forceinline__ bf16x8 frag(const lds_char* t, int r, int s, int kg) {
    return *reinterpret_cast<const __attribute__((address_space(3))) bf16x8*>(t + koff(r, 2 * s + kg));
  }
};

// ------------------------------------------------------- N-major operand
// Stored [k][cols] with the tile index contiguous: element (k, c) at byte
// k*ld + 2c of the sub-tile's base.  The tile's 256 columns are two
// sub-tiles of 128 (sub-tile j starts at ptr_j, has cols_j valid columns and
// range_j readable bytes); k < kmax valid.  Loads move half a step (32 k)
// at a time (the load stream below).  LDS per half: two sub-tiles [32 k][128
// cols] bf16, 256-byte
// rows, 16-byte chunk c of row k at ((c ^ (4 (k & 3))) << 4): the 32 lanes of
// one ds_read_b64_tr_b16 pass (4 rows x 4 chunks x 2 halves) hit all 64 banks.
__device__ __forceinline__ int noff(int k, int col) {
  return k * 256 + ((((col >> 3) ^ (4 * (k & 3)))) << 4) + ((col >> 2) & 1) * 8;
}

struct NOperand {
  const uint16_t* ptr0;
  const uint16_t* ptr1;
  int64_t range0, range1;
  uint32_t ld;
  int cols0, cols1;
  int kmax;
  // MFMA fragment of tile column block c0 (multiple of 32) from one half:
  // lane l gets 8 consecutive k (k-group l/32 of substep s, 0..1, of the
  // half) of column c0 + l%32, built from two transposing reads of 4 k each.
  static __device__ __forceinline__ bf16x8 frag(const lds_char* t, int c0, int s, int lane) {
    const int g = lane >> 4, r = lane & 15;
    const int st = c0 >> 7;
    const int col = (c0 & 127) + 16 * (g & 1) + 4 * (r & 3);
    const int k = 16 * s + 8 * (g >> 1) + (r >> 2);
    const lds_char* b = t + st * (HALF / 2);
    const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(b + noff(k, col)));
    const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4*)(b + noff(k + 4, col)));
    typedef short s16x8 __attribute__((ext_vector_type(8)));
    const s16x8 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
  }
};

// ------------------------------------------------- per-tile load streams
// The loads of one operand of one tile, prepared once when the tile starts,
// so that a K step's loads cost a source pick, an offset add and the loads
// themselves.  Any step can be issued in any order (nothing advances per
// issue).  NL waves (8: all of them, or 4: one group of the ping-pong
// schedule) load one operand; `wave` is a wave's rank among them.

// K-contiguous operand.  Load q (0 .. LK - 1) of wave w, I = LK w + q, fills
// tile rows 8 I .. 8 I + 7: lane l takes row 8 I + l / 8 and the 16-byte
// chunk lc = (l % 8) ^ ((row / 2) % 8), which is lc0 for even q and lc0 ^ 4
// for odd q.  A lane whose row lies past the tile's valid rows gets an
// offset past every descriptor range (it reads zeros); only a step that
// reaches past the valid k masks chunks.  DUALK: steps [0, nk0) read source
// 0, the rest source 1 (k restarting at 0).
template <bool DUALK, int NL>
struct KStream {
  static constexpr int LK = UNIT / 1024 / NL;  // 16-byte direct loads per lane and step
  i32x4 rs0, rs1;
  uint32_t voff[LK];  // lane offset of load q at k = 0
  int nk0, km0, km1;
  __device__ __forceinline__ void setup(const KOperand& op, int wave, int lane) {
    rs0 = op.rsrc0;
    rs1 = op.rsrc1;
    nk0 = op.nk0;
    km0 = op.kmax0;
    km1 = op.kmax1;
    const int rl = lane >> 3;
    const int lc0 = (lane & 7) ^ (lane >> 4);
#pragma unroll
    for (int q = 0; q < LK; ++q) {
      const int row = (wave * LK + q) * 8 + rl;
      const int lc = (q & 1) ? (lc0 ^ 4) : lc0;
      voff[q] = row < op.rows ? static_cast<uint32_t>(row) * op.ld + static_cast<uint32_t>(lc * 16)
                              : OOB;
    }
  }
  // step j of the tile into the LDS unit at `u`
  __device__ __forceinline__ void issue(int j, uint32_t u, int wave) const {
    const bool s1 = DUALK && j >= nk0;
    const int k0 = (s1 ? j - nk0 : j) * BK;
    const int km = s1 ? km1 : km0;
    const i32x4 rs = s1 ? rs1 : rs0;
    const uint32_t kb = static_cast<uint32_t>(k0) * 2u;
    if (k0 + BK <= km) {
#pragma unroll
      for (int q = 0; q < LK; ++q) load_lds16(rs, voff[q] + kb, u + (wave * LK + q) * 1024);
    } else {
      const int lane = opaque(static_cast<int>(threadIdx.x & 63));
      const int lc0 = (lane & 7) ^ (lane >> 4);
#pragma unroll
      for (int q = 0; q < LK; ++q) {
        const int lc = (q & 1) ? (lc0 ^ 4) : lc0;
        load_lds16(rs, k0 + lc * 8 < km ? voff[q] + kb : OOB, u + (wave * LK + q) * 1024);
      }
    }
  }
  // the same number of loads, all out of range (zeros into an unused slot)
  static __device__ __forceinline__ void none(const i32x4& nil, uint32_t u, int wave) {
#pragma unroll
    for (int q = 0; q < LK; ++q) load_lds16(nil, OOB, u + (wave * LK + q) * 1024);
  }
};

// N-contiguous operand: this wave's sub-tile of 128 columns (the first half
// of the loading waves load sub-tile 0, the second half sub-tile 1).  Half h
// (0, 1) of step j covers rows r0 = 64 j + 32 h .. r0 + 31; load Q (0 ..
// LH - 1), I = LH w + Q, covers rows r0 + kr .. +3, kr = 4 (I % 8): lane l
// takes row r0 + kr + l / 16 and column 8 ((l % 16) ^ (4 (l / 16))).  The
// descriptor's base moves to row r0 (64-bit, so lane offsets stay below 32
// rows at any K) while its range stays the bound set at the tile's start:
// every lane's column and row are checked, so valid lanes never reach it.
// Lanes of columns past the sub-tile's valid columns get an out-of-range
// offset; only a half that reaches past the valid k masks rows.
template <int NL>
struct NStream {
  static constexpr int LH = HALF / 1024 / NL;  // 16-byte direct loads per lane and half step
  uint64_t base;       // byte address of the sub-tile's row 0
  uint32_t range, ld;  // descriptor range from row 0; row pitch in bytes
  uint32_t voff[LH];   // lane offset of load Q from the half's first row
  int kmax;
  __device__ __forceinline__ void setup(const NOperand& op, int wave, int lane) {
    const int sub = (wave * LH) >> 3;
    const i32x4 r = make_rsrc(sub ? op.ptr1 : op.ptr0, sub ? op.range1 : op.range0);
    base = (static_cast<uint64_t>(static_cast<uint32_t>(r[1]) & 0xffffu) << 32) |
           static_cast<uint32_t>(r[0]);
    range = static_cast<uint32_t>(r[2]);
    ld = op.ld;
    kmax = op.kmax;
    const int kl = lane >> 4;
    const int col = ((lane & 15) ^ (4 * kl)) * 8;
    const int cols = sub ? op.cols1 : op.cols0;
#pragma unroll
    for (int q = 0; q < LH; ++q) {
      const int kr = ((wave * LH + q) & 7) * 4;
      voff[q] = col < cols ? static_cast<uint32_t>(kr + kl) * ld + static_cast<uint32_t>(col * 2)
                           : OOB;
    }
  }
  // half h of step j into the LDS half at `u` (both sub-tiles' halves)
  __device__ __forceinline__ void issue(int j, int h, uint32_t u, int wave) const {
    const int sub = (wave * LH) >> 3;
    const int r0 = j * BK + h * (BK / 2);
    const uint64_t a = base + static_cast<uint64_t>(static_cast<uint32_t>(r0)) * ld;
    i32x4 rs;
    rs[0] = static_cast<int>(a & 0xffffffffu);
    rs[1] = static_cast<int>((a >> 32) & 0xffffu);
    rs[2] = static_cast<int>(range);
    rs[3] = 0x00020000;
    const int krem = kmax - r0;
    if (krem >= BK / 2) {
#pragma unroll
      for (int q = 0; q < LH; ++q) {
        const int I = wave * LH + q;
        load_lds16(rs, voff[q], u + sub * (HALF / 2) + (I & 7) * 1024);
      }
    } else {
      const int kl = opaque(static_cast<int>(threadIdx.x & 63)) >> 4;
#pragma unroll
      for (int q = 0; q < LH; ++q) {
        const int I = wave * LH + q;
        const int kr = (I & 7) * 4;
        load_lds16(rs, kl < krem - kr ? voff[q] : OOB, u + sub * (HALF / 2) + (I & 7) * 1024);
      }
    }
  }
  static __device__ __forceinline__ void none(const i32x4& nil, uint32_t u, int wave) {
#pragma unroll
    for (int q = 0; q < LH; ++q) {
      const int I = wave * LH + q;
      load_lds16(nil, OOB, u + (I >> 3) * (HALF / 2) + (I & 7) * 1024);
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
  const int32_t* wk_start;  // [E_loc+1] prefix of per-expert K steps (weight gradients)
  const int32_t* nz_start;  // [E_loc+1] prefix of the count of experts with rows
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
  // dense products
  const uint16_t* da;       // operand A
  const uint16_t* db;       // operand B
  void* dc;                 // output
  const int32_t* target;    // vocabulary: target of each row [N]
  const float* lse;         // vocabulary: log-sum-exp of each row [N]
  const float* dloss;       // vocabulary: upstream gradient of each row [N]
  float* yt;                // vocabulary: target logit of each row [N]
  int64_t a_ld, b_ld, c_ld; // row pitches (elements)
  int64_t c_bstride;        // output elements per batch
  int64_t v0;               // vocabulary: block's first column in B's (or dW's) row
  int dM, dN, dK;           // output rows, valid output columns, contraction length
  int kspan, batches;       // contraction rows per batch, batches
  int64_t bc0;              // vocabulary: B's first column (the block, or 0 when staged)
  int64_t cc0;              // vocabulary: dW's first column (VOC_DW)
  int dE;                   // router: experts (the lo parts sit 2E columns into DL3)
  int flag;                 // RT_DX: add to dx; VOC_DX: first block (store, no add)
};

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
//  * Weight gradients: every expert with rows has MT x NT tiles of K = its
//    row count; the tiles (expert-major, row tiles of one column tile
//    adjacent) are cut into 8 contiguous ranges of equal K-step work, one per
//    XCD, dealt round-robin to the XCD's CUs.  An expert's tiles thus share
//    one L2 (its activations and gradient rows are fetched once per XCD)
//    unless it is larger than an XCD's share.
// Schedule tables of one launch, read with scalar loads: tile decoding is
// uniform, and a scalar load waits on the LDS/scalar counter only, never on
// the vector-memory counter that tracks the operand loads in flight.
__device__ __forceinline__ int sld(const int32_t* p) {
  int v;
  asm volatile("s_load_dword %0, %1, 0x0\n\ts_waitcnt lgkmcnt(0)" : "=s"(v) : "s"(p) : "memory");
  return v;
}
struct Tables {
  const int32_t* mt_start_;  // [E_loc + 1]
  const int32_t* offsets_;   // [E_loc + 1]
  const int32_t* wk_start_;  // [E_loc + 1]
  const int32_t* nz_start_;  // [E_loc + 1]
  __device__ __forceinline__ int mt(int i) const { return sld(mt_start_ + i); }
  __device__ __forceinline__ int off(int i) const { return sld(offsets_ + i); }
  __device__ __forceinline__ int wk(int i) const { return sld(wk_start_ + i); }
  __device__ __forceinline__ int nz(int i) const { return sld(nz_start_ + i); }
};

// Position (m, n) of tile `local` of an mt x nt grid, walked in groups of
// GM row tiles: inside a group the row tiles of one column tile are
// adjacent and the group's column tiles follow one another.  The 32
// consecutive tiles an XCD runs at a time then form a GM x 32/GM block
// that shares GM row slabs and 32/GM column slabs of the operands in that
// XCD's L2 (instead of 32 row slabs and one column slab).  Measured best:
// GM = 4 for the row-grouped products (4 row slabs of activations, 8
// column slabs of an expert's weights), GM = 8 for the weight gradients and
// the dense products.
template <int GM>
__device__ __forceinline__ void tile_pos(int local, int mt, int nt, int& m, int& n) {
  const int per = GM * nt;
  const int grp = local / per;
  const int r = local - grp * per;
  const int gm = min(GM, mt - grp * GM);
  m = grp * GM + r % gm;
  n = r / gm;
}

template <int MODE>
struct TileIter {
  static constexpr bool WG = Traits<MODE>::WG;
  static constexpr bool DUAL = Traits<MODE>::DUAL;
  static constexpr bool DENSE = Traits<MODE>::DENSE;
  int xcd, j, cpx, i;
  int total, end;  // row-grouped: tile count, end of this XCD's range
  int unit;        // weight gradients: tiles per expert with rows (MT * NT)
  int ecache;      // weight gradients: expert of the previous tile
  bool zeros;      // weight gradients: visit only the tiles of experts without rows

  // Weight gradients: first tile whose K-step work starts at or after `b`.
  __device__ __forceinline__ int wg_tile_at(const GemmArgs& g, const Tables& tb, int64_t b) const {
    const int64_t W = static_cast<int64_t>(unit) * tb.wk(g.E_loc);
    if (b >= W) return unit * tb.nz(g.E_loc);
    int lo = 0, hi = g.E_loc - 1;  // smallest e with unit * wk(e + 1) > b
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if (static_cast<int64_t>(unit) * tb.wk(mid + 1) > b) hi = mid; else lo = mid + 1;
    }
    const int64_t w0 = static_cast<int64_t>(unit) * tb.wk(lo);
    const int nk = tb.wk(lo + 1) - tb.wk(lo);
    return unit * tb.nz(lo) + static_cast<int>((b - w0 + nk - 1) / nk);
  }

  __device__ __forceinline__ void init(const GemmArgs& g, const Tables& tb, bool zero_tiles = false) {
    zeros = zero_tiles;
    cpx = gridDim.x / NXCD;
    xcd = blockIdx.x % NXCD;
    j = blockIdx.x / NXCD;
    i = 0;
    if constexpr (DENSE) {
      // batches x MT x NT tiles, row tiles of one column tile adjacent, cut
      // into 8 contiguous equal ranges (one per XCD)
      total = g.batches * g.MT * g.NT;
      const int per = (total + NXCD - 1) / NXCD;
      end = min((xcd + 1) * per, total);
      total = xcd * per;
    } else if constexpr (!WG) {
      total = tb.mt(g.E_loc) * g.NT;
      const int per = (total + NXCD - 1) / NXCD;
      end = min((xcd + 1) * per, total);
      total = xcd * per;  // start of this XCD's range
    } else if (!zero_tiles) {
      unit = g.MT * g.NT;
      ecache = 0;
      const int64_t W = static_cast<int64_t>(unit) * tb.wk(g.E_loc);
      total = wg_tile_at(g, tb, W * xcd / NXCD);
      end = wg_tile_at(g, tb, W * (xcd + 1) / NXCD);
    }
  }
  __device__ __forceinline__ Tile next(const GemmArgs& g, const Tables& tb) {
    Tile t;
    t.valid = false;
    if constexpr (DENSE) {
      const int L = total + j + cpx * i;
      ++i;
      if (L >= end) return t;
      const int per_b = g.MT * g.NT;
      const int b = L / per_b, local = L - b * per_b;
      t.e = b;
      int tm, tn;
      tile_pos<8>(local, g.MT, g.NT, tm, tn);
      t.m0 = tm * BM;
      t.n0 = tn * (DUAL ? BN / 2 : BN);
      t.seg = b * g.kspan;               // first contraction row of the batch
      t.ne = min(g.kspan, g.dK - t.seg);  // its contraction rows
      t.nk = (t.ne + BK - 1) / BK;
      t.valid = true;
      return t;
    } else if constexpr (!WG) {
      const int L = total + j + cpx * i;
      ++i;
      if (L >= end) return t;
      int lo = 0, hi = g.E_loc;
      while (hi - lo > 1) {
        const int mid = (lo + hi) >> 1;
        if (tb.mt(mid) * g.NT <= L) lo = mid; else hi = mid;
      }
      t.e = __builtin_amdgcn_readfirstlane(lo);
      const int ms0 = tb.mt(lo);
      const int mt_e = tb.mt(lo + 1) - ms0;
      const int local = L - ms0 * g.NT;
      int tm, tn;
      tile_pos<4>(local, mt_e, g.NT, tm, tn);
      t.m0 = tm * BM;
      t.n0 = tn * (DUAL ? BN / 2 : BN);
      t.seg = tb.off(lo);
      t.ne = tb.off(lo + 1) - t.seg;
      const int K = (MODE == FWD_GATE_UP || MODE == DGRAD_DOWN) ? g.d : g.f;
      t.nk = ((K + BK - 1) / BK) * (MODE == DGRAD_GATE_UP ? 2 : 1);
      t.valid = true;
      return t;
    } else if (!zeros) {
      const int L = total + j + cpx * i;
      ++i;
      if (L >= end) return t;
      int e = ecache;  // usually the previous tile's expert
      if (!(unit * tb.nz(e) <= L && L < unit * tb.nz(e + 1))) {
        int lo = 0, hi = g.E_loc - 1;  // smallest e with unit * nz(e + 1) > L
        while (lo < hi) {
          const int mid = (lo + hi) >> 1;
          if (unit * tb.nz(mid + 1) > L) hi = mid; else lo = mid + 1;
        }
        e = lo;
      }
      ecache = e;
      t.e = __builtin_amdgcn_readfirstlane(e);
      const int local = L - unit * tb.nz(e);
      int tm, tn;
      tile_pos<8>(local, g.MT, g.NT, tm, tn);
      t.m0 = tm * BM;
      t.n0 = tn * (DUAL ? BN / 2 : BN);
      t.seg = tb.off(e);
      t.ne = tb.off(e + 1) - t.seg;
      t.nk = (t.ne + BK - 1) / BK;
      t.valid = true;
      return t;
    } else {
      // experts without rows: every one of their tiles, dealt over the grid
      while (true) {
        const int G = blockIdx.x + gridDim.x * i;
        ++i;
        if (G >= g.E_loc * g.MT * g.NT) return t;
        const int e = G / (g.MT * g.NT), local = G % (g.MT * g.NT);
        if (tb.off(e + 1) != tb.off(e)) continue;
        t.e = __builtin_amdgcn_readfirstlane(e);
        t.m0 = (local % g.MT) * BM;
        t.n0 = (local / g.MT) * (DUAL ? BN / 2 : BN);
        t.seg = tb.off(e);
        t.ne = 0;
        t.nk = 0;
        t.valid = true;
        return t;
      }
    }
  }
};

template <int MODE>
__global__ __launch_bounds__(NTHR, 1) void grouped_gemm_kernel(GemmArgs g) {
  __shared__ __align__(1024) char lds[NRING * UNIT];
  constexpr bool WGRAD = Traits<MODE>::WG;
  constexpr bool DENSE = Traits<MODE>::DENSE;
  constexpr bool DUAL = Traits<MODE>::DUAL;
  constexpr bool A_N = Traits<MODE>::A_N;  // A side N-major?
  constexpr bool B_K = Traits<MODE>::B_K;  // B side K-major?
  using AOp = typename std::conditional<A_N, NOperand, KOperand>::type;
  using BOp = typename std::conditional<B_K, KOperand, NOperand>::type;

  const int d = g.d, f = g.f;
  const int64_t wdf = static_cast<int64_t>(d) * f;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = w & 1, wn = w >> 1;  // 2 x 4 waves, each 128 rows x 64 columns
  const int l32 = lane & 31, lh = lane >> 5;

  // ------------------------------------------------------- operand setup
  // A side = rows m of the output, B side = columns n of the output.
  auto setupA = [&](const Tile& tl, AOp& A) __attribute__((always_inline)) {
    const int m0 = tl.m0, seg = tl.seg, ne = tl.ne;
    if constexpr (MODE == FWD_GATE_UP) {
      const uint16_t* xa = g.x_perm + (int64_t)(seg + m0) * d;
      A.rsrc0 = A.rsrc1 = make_rsrc(xa, (int64_t)(ne - m0) * d * 2);
      A.ld = d * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = d; A.nk0 = (d + BK - 1) / BK;
    } else if constexpr (MODE == FWD_DOWN) {
      const uint16_t* aa = g.act_in + (int64_t)(seg + m0) * f;
      A.rsrc0 = A.rsrc1 = make_rsrc(aa, (int64_t)(ne - m0) * f * 2);
      A.ld = f * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = f; A.nk0 = (f + BK - 1) / BK;
    } else if constexpr (MODE == DGRAD_DOWN) {
      const uint16_t* ya = g.dy + (int64_t)(seg + m0) * d;
      A.rsrc0 = A.rsrc1 = make_rsrc(ya, (int64_t)(ne - m0) * d * 2);
      A.ld = d * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = d; A.nk0 = (d + BK - 1) / BK;
    } else if constexpr (MODE == DGRAD_GATE_UP) {
      const int64_t ro = (int64_t)(seg + m0) * f;
      A.rsrc0 = make_rsrc(g.dhg_in + ro, (int64_t)(ne - m0) * f * 2);
      A.rsrc1 = make_rsrc(g.dhu_in + ro, (int64_t)(ne - m0) * f * 2);
      A.ld = f * 2; A.rows = ne - m0; A.kmax0 = A.kmax1 = f; A.nk0 = (f + BK - 1) / BK;
    } else if constexpr (MODE == WGRAD_GATE_UP) {
      A.ptr0 = g.x_perm + (int64_t)seg * d + m0; A.range0 = ((int64_t)ne * d - m0) * 2;
      A.ptr1 = A.ptr0 + 128; A.range1 = A.range0 - 256;
      A.ld = d * 2; A.cols0 = d - m0; A.cols1 = d - m0 - 128; A.kmax = ne;
    } else if constexpr (MODE == WGRAD_DOWN) {
      A.ptr0 = g.act_in + (int64_t)seg * f + m0; A.range0 = ((int64_t)ne * f - m0) * 2;
      A.ptr1 = A.ptr0 + 128; A.range1 = A.range0 - 256;
      A.ld = f * 2; A.cols0 = f - m0; A.cols1 = f - m0 - 128; A.kmax = ne;
    } else if constexpr (A_N) {
      // RT_DW: X [T][d], contraction rows = the batch's tokens;
      // VOC_DW: X [N][H], contraction rows = all N tokens (seg = 0)
      A.ptr0 = g.da + seg * g.a_ld + m0; A.range0 = ((int64_t)ne * g.a_ld - m0) * 2;
      A.ptr1 = A.ptr0 + 128; A.range1 = A.range0 - 256;
      A.ld = static_cast<uint32_t>(g.a_ld * 2); A.cols0 = g.dM - m0; A.cols1 = g.dM - m0 - 128;
      A.kmax = ne;
    } else {
      // K-contiguous dense A: RT_DX DL3 [T][E3p]; VOC_FWD/GRAD X [N][H];
      // VOC_DX G [N][gp] from column seg (the batch's share of the block)
      const uint16_t* aa = g.da + (int64_t)m0 * g.a_ld + seg;
      A.rsrc0 = A.rsrc1 = make_rsrc(aa, ((int64_t)(g.dM - m0) * g.a_ld - seg) * 2);
      A.ld = static_cast<uint32_t>(g.a_ld * 2); A.rows = g.dM - m0;
      A.kmax0 = A.kmax1 = ne; A.nk0 = (ne + BK - 1) / BK;
    }
  };
  auto setupB = [&](const Tile& tl, BOp& B) __attribute__((always_inline)) {
    const int e = tl.e, n0 = tl.n0, seg = tl.seg, ne = tl.ne;
    if constexpr (MODE == FWD_GATE_UP) {
      B.ptr0 = g.wg + e * wdf + n0; B.range0 = (wdf - n0) * 2;
      B.ptr1 = g.wu + e * wdf + n0; B.range1 = (wdf - n0) * 2;
      B.ld = f * 2; B.cols0 = B.cols1 = f - n0; B.kmax = d;
    } else if constexpr (MODE == FWD_DOWN) {
      B.ptr0 = g.wd + e * wdf + n0; B.range0 = (wdf - n0) * 2;
      B.ptr1 = B.ptr0 + 128; B.range1 = (wdf - n0 - 128) * 2;
      B.ld = d * 2; B.cols0 = d - n0; B.cols1 = d - n0 - 128; B.kmax = f;
    } else if constexpr (MODE == DGRAD_DOWN) {
      const uint16_t* wb = g.wd + e * wdf + (int64_t)n0 * d;
      B.rsrc0 = B.rsrc1 = make_rsrc(wb, (int64_t)(f - n0) * d * 2);
      B.ld = d * 2; B.rows = f - n0; B.kmax0 = B.kmax1 = d; B.nk0 = (d + BK - 1) / BK;
    } else if constexpr (MODE == DGRAD_GATE_UP) {
      const int64_t wo = e * wdf + (int64_t)n0 * f;
      B.rsrc0 = make_rsrc(g.wg + wo, (int64_t)(d - n0) * f * 2);
      B.rsrc1 = make_rsrc(g.wu + wo, (int64_t)(d - n0) * f * 2);
      B.ld = f * 2; B.rows = d - n0; B.kmax0 = B.kmax1 = f; B.nk0 = (f + BK - 1) / BK;
    } else if constexpr (MODE == WGRAD_GATE_UP) {
      B.ptr0 = g.dhg_in + (int64_t)seg * f + n0; B.range0 = ((int64_t)ne * f - n0) * 2;
      B.ptr1 = g.dhu_in + (int64_t)seg * f + n0; B.range1 = B.range0;
      B.ld = f * 2; B.cols0 = B.cols1 = f - n0; B.kmax = ne;
    } else if constexpr (MODE == WGRAD_DOWN) {
      B.ptr0 = g.dy + (int64_t)seg * d + n0; B.range0 = ((int64_t)ne * d - n0) * 2;
      B.ptr1 = B.ptr0 + 128; B.range1 = B.range0 - 256;
      B.ld = d * 2; B.cols0 = d - n0; B.cols1 = d - n0 - 128; B.kmax = ne;
    } else if constexpr (MODE == RT_DW) {
      // DL3 [T][E3p] = [hi | hi | lo]: sub-tile 0 from the first hi group,
      // sub-tile 1 from the lo group, the same 128 experts
      const uint16_t* r0 = g.db + seg * g.b_ld;
      B.ptr0 = r0 + n0; B.range0 = ((int64_t)ne * g.b_ld - n0) * 2;
      B.ptr1 = r0 + 2 * g.dE + n0; B.range1 = ((int64_t)ne * g.b_ld - 2 * g.dE - n0) * 2;
      B.ld = static_cast<uint32_t>(g.b_ld * 2); B.cols0 = B.cols1 = g.dN - n0; B.kmax = ne;
    } else if constexpr (MODE == VOC_DX) {
      // W [H][ldw], K-contiguous rows h, the block's columns from bc0 + seg
      const uint16_t* wb = g.db + (int64_t)n0 * g.b_ld + g.bc0 + seg;
      B.rsrc0 = B.rsrc1 = make_rsrc(wb, ((int64_t)(g.dN - n0) * g.b_ld - g.bc0 - seg) * 2);
      B.ld = static_cast<uint32_t>(g.b_ld * 2); B.rows = g.dN - n0;
      B.kmax0 = B.kmax1 = ne; B.nk0 = (ne + BK - 1) / BK;
    } else {
      // N-contiguous dense B: RT_DX W3 [3E][d] (bc0 = 0); VOC_FWD/GRAD W
      // [H][ldw] from column bc0 (the block); VOC_DW G [N][gp] (bc0 = 0)
      const int64_t c0 = g.bc0;
      const uint16_t* bb = g.db + c0 + seg * g.b_ld;
      B.ptr0 = bb + n0; B.range0 = ((int64_t)ne * g.b_ld - c0 - n0) * 2;
      B.ptr1 = B.ptr0 + 128; B.range1 = B.range0 - 256;
      B.ld = static_cast<uint32_t>(g.b_ld * 2); B.cols0 = g.dN - n0; B.cols1 = g.dN - n0 - 128;
      B.kmax = ne;
    }
  };

  // First tile row of each 32-row MFMA block: four on the A side, two on
  // the B side (dual: the gate and the up column block of the same f).
  int arow[4], brow[2];
#pragma unroll
  for (int i = 0; i < 4; ++i) arow[i] = wm * 128 + 32 * i;
#pragma unroll
  for (int jj = 0; jj < 2; ++jj) brow[jj] = DUAL ? jj * (BN / 2) + wn * 32 : wn * 64 + 32 * jj;

  f32x16 acc[4][2];
  auto zero_acc = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int jj = 0; jj < 2; ++jj)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][jj][r] = 0.0f;
  };

  // ------------------------------------------------------------ epilogue
  // acc[i][j][4q + u]: output row m = arow[i] + l32 (tile-relative),
  // output column n = brow[j] + 8q + 4*lh + u.  Each wave passes its
  // 128 x 64 block through its own 4 KiB LDS patch, 32 rows (16 in fp32) at
  // a time: it writes the accumulators in the MFMA layout and reads them
  // back row-major, so that every global access moves 16 bytes per lane and
  // 4 or 8 lanes cover one contiguous row segment (whole 64- or 128-byte
  // pieces instead of 32 scattered 8-byte pieces per instruction).  Patch
  // chunks carry XOR swizzles that keep the 64 banks conflict-free.
  auto epilogue = [&](const Tile& tl, lds_char* patch) __attribute__((always_inline)) {
    const int e = tl.e, m0 = tl.m0, n0 = tl.n0, seg = tl.seg, ne = tl.ne;
    // lane-derived indices recomputed here (not hoisted and kept live
    // across the K loop, where they would be spilled)
    const int lane = opaque(threadIdx.x & 63);
    const int l32 = lane & 31, lh = lane >> 5;
    const int mvalid = DENSE   ? (g.dM - m0)
                       : WGRAD ? ((MODE == WGRAD_GATE_UP ? d : f) - m0)
                               : (ne - m0);
    typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
    typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
    typedef float f32x4v __attribute__((ext_vector_type(4)));
    auto put8 = [&](int off, uint2 v) __attribute__((always_inline)) {
      *(__attribute__((address_space(3))) u32x2v*)(patch + off) = u32x2v{v.x, v.y};
    };
    auto put16 = [&](int off, float4 v) __attribute__((always_inline)) {
      *(__attribute__((address_space(3))) f32x4v*)(patch + off) = f32x4v{v.x, v.y, v.z, v.w};
    };
    auto get16 = [&](int off) __attribute__((always_inline)) {
      const u32x4v v = *(__attribute__((address_space(3))) u32x4v*)(patch + off);
      return make_uint4(v[0], v[1], v[2], v[3]);
    };
    auto getf16 = [&](int off) __attribute__((always_inline)) {
      const f32x4v v = *(__attribute__((address_space(3))) f32x4v*)(patch + off);
      return make_float4(v[0], v[1], v[2], v[3]);
    };
    auto fence = []() __attribute__((always_inline)) { asm volatile("" ::: "memory"); };
    // rows 16..31 of a bf16 patch hold their two 8-byte halves swapped
    auto unswap = [](uint4 v, int r) __attribute__((always_inline)) {
      return (r & 16) ? make_uint4(v.z, v.w, v.x, v.y) : v;
    };
    static_for<4>([&](auto I) {
      constexpr int i = I;
      const int rb = wm * 128 + 32 * i;  // tile row of the block's first row
      if (rb >= mvalid) return;
      if constexpr (MODE == FWD_GATE_UP || MODE == WGRAD_GATE_UP) {
        // gate [32][32] bf16 at +0, up at +2048; 64-byte rows, 16-byte chunk c
        // of row r at c ^ ((r / 4) % 4)
        static_for<4>([&](auto Q) {
          constexpr int q = Q;
          const int off = l32 * 64 + ((q ^ ((l32 >> 2) & 3)) << 4) + ((lh ^ (l32 >> 4)) & 1) * 8;
          put8(off, pack4(acc[i][0][4 * q], acc[i][0][4 * q + 1], acc[i][0][4 * q + 2], acc[i][0][4 * q + 3]));
          put8(2048 + off, pack4(acc[i][1][4 * q], acc[i][1][4 * q + 1], acc[i][1][4 * q + 2],
                                 acc[i][1][4 * q + 3]));
        });
        fence();
        static_for<2>([&](auto Tt) {
          constexpr int t = Tt;
          const int r = 16 * t + (lane >> 2), c = lane & 3;
          const int off = r * 64 + ((c ^ ((r >> 2) & 3)) << 4);
          const uint4 hgv = unswap(get16(off), r), huv = unswap(get16(2048 + off), r);
          const int rt = rb + r, col = n0 + wn * 32 + 8 * c;
          if (rt < mvalid && col < f) {
            if constexpr (MODE == FWD_GATE_UP) {
              const int64_t o = (int64_t)(seg + m0 + rt) * f + col;
              const uint32_t gw[4] = {hgv.x, hgv.y, hgv.z, hgv.w};
              const uint32_t uw[4] = {huv.x, huv.y, huv.z, huv.w};
              uint32_t aw[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                const float g0 = bf16_lo(gw[u]), g1 = bf16_hi(gw[u]);
                aw[u] = pack_bf16x2(g0 * sigmoidf_fast(g0) * bf16_lo(uw[u]),
                                    g1 * sigmoidf_fast(g1) * bf16_hi(uw[u]));
              }
              *reinterpret_cast<uint4*>(g.hg + o) = hgv;
              *reinterpret_cast<uint4*>(g.hu + o) = huv;
              *reinterpret_cast<uint4*>(g.act + o) = make_uint4(aw[0], aw[1], aw[2], aw[3]);
            } else {
              const int64_t o = e * wdf + (int64_t)(m0 + rt) * f + col;
              *reinterpret_cast<uint4*>(g.dwg + o) = hgv;
              *reinterpret_cast<uint4*>(g.dwu + o) = huv;
            }
          }
        });
        fence();
      } else if constexpr (MODE == DGRAD_DOWN) {
        // SwiGLU backward from the fp32 dA block, 16 rows at a time:
        // [16][64] fp32, 256-byte rows, 16-byte chunk c of row r at c ^ r.
        // Its inputs for the block's 32 rows come in one batch; rows past the
        // segment read as zero.
        const int cg = lane & 7;
        const int col = n0 + wn * 64 + 8 * cg;
        u32x4a hgq[4], huq[4];
        {
          const int64_t rbase = (int64_t)(seg + m0) * f;
          const int64_t rbytes = (int64_t)(ne - m0) * f * 2;
          const i32x4 rhg = make_rsrc(g.hg_in + rbase, rbytes), rhu = make_rsrc(g.hu_in + rbase, rbytes);
          uint32_t off[4];
          static_for<4>([&](auto Tt) {  // Tt = 2 h + t
            constexpr int ht = Tt;
            const int rt = rb + 16 * (ht / 2) + 8 * (ht % 2) + (lane >> 3);
            off[ht] = col < f ? static_cast<uint32_t>((rt * f + col) * 2) : OOB;
          });
          load_2x4_wait(rhg, rhu, off, hgq, huq);
        }
        static_for<2>([&](auto H) {
          constexpr int h = H;
          if ((l32 >> 4) == h) {
            const int rr = l32 & 15;
            static_for<2>([&](auto J) {
              static_for<4>([&](auto Q) {
                constexpr int j = J, q = Q;
                const int c = 8 * j + 2 * q + lh;
                put16(rr * 256 + ((c ^ rr) << 4),
                      make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                  acc[i][j][4 * q + 3]));
              });
            });
          }
          fence();
          static_for<2>([&](auto Tt) {
            constexpr int t = Tt;
            const int rr = 8 * t + (lane >> 3);
            const float4 d0 = getf16(rr * 256 + (((2 * cg) ^ rr) << 4));
            const float4 d1 = getf16(rr * 256 + (((2 * cg + 1) ^ rr) << 4));
            const int rt = rb + 16 * h + rr;
            const u32x4a hq = hgq[2 * h + t], uq = huq[2 * h + t];
            {  // computed in every lane (the loads above always complete), stored where valid
              const float da[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
              const uint32_t gw[4] = {hq[0], hq[1], hq[2], hq[3]};
              const uint32_t uw[4] = {uq[0], uq[1], uq[2], uq[3]};
              uint32_t dgw[4], duw[4], aw[4];
#pragma unroll
              for (int u = 0; u < 4; ++u) {
                float dg[2], du[2], av[2];
#pragma unroll
                for (int v = 0; v < 2; ++v) {
                  const float gz = v ? bf16_hi(gw[u]) : bf16_lo(gw[u]);
                  const float uz = v ? bf16_hi(uw[u]) : bf16_lo(uw[u]);
                  const float sg = sigmoidf_fast(gz);
                  const float sl = gz * sg;
                  dg[v] = da[2 * u + v] * uz * (sg + sl * (1.0f - sg));
                  du[v] = da[2 * u + v] * sl;
                  av[v] = sl * uz;
                }
                dgw[u] = pack_bf16x2(dg[0], dg[1]);
                duw[u] = pack_bf16x2(du[0], du[1]);
                aw[u] = pack_bf16x2(av[0], av[1]);
              }
              if (rt < mvalid && col < f) {
                const int64_t o = (int64_t)(seg + m0 + rt) * f + col;
                *reinterpret_cast<uint4*>(g.dhg + o) = make_uint4(dgw[0], dgw[1], dgw[2], dgw[3]);
                *reinterpret_cast<uint4*>(g.dhu + o) = make_uint4(duw[0], duw[1], duw[2], duw[3]);
                *reinterpret_cast<uint4*>(g.act + o) = make_uint4(aw[0], aw[1], aw[2], aw[3]);
              }
            }
          });
          fence();
        });
      } else if constexpr (MODE == RT_DW) {
        // fp32 partial dW_r of the batch: hi and lo sums of one expert column
        // added, straight from the accumulators (4 consecutive columns per
        // lane and row)
        if (rb + l32 < mvalid) {
          float* out = static_cast<float*>(g.dc) + (int64_t)e * g.c_bstride +
                       (int64_t)(m0 + rb + l32) * g.c_ld;
          static_for<4>([&](auto Q) {
            constexpr int q = Q;
            const int col = n0 + wn * 32 + 8 * q + 4 * lh;
            const float v0 = acc[i][0][4 * q] + acc[i][1][4 * q];
            const float v1 = acc[i][0][4 * q + 1] + acc[i][1][4 * q + 1];
            const float v2 = acc[i][0][4 * q + 2] + acc[i][1][4 * q + 2];
            const float v3 = acc[i][0][4 * q + 3] + acc[i][1][4 * q + 3];
            if (col + 4 <= g.dN && (g.c_ld & 3) == 0) {
              *reinterpret_cast<float4*>(out + col) = make_float4(v0, v1, v2, v3);
            } else {
              if (col < g.dN) out[col] = v0;
              if (col + 1 < g.dN) out[col + 1] = v1;
              if (col + 2 < g.dN) out[col + 2] = v2;
              if (col + 3 < g.dN) out[col + 3] = v3;
            }
          });
        }
      } else if constexpr (MODE == VOC_FWD) {
        // Per row, the (max, sum of exp(y - max)) of this wave's 64 block
        // columns (lanes l and l + 32 hold 32 each), and the target's logit
        // where this wave holds the target column.
        const int rt = rb + l32;
        const bool rok = rt < mvalid;
        const int64_t row = (int64_t)m0 + rt;
        const int cb = n0 + wn * 64;  // block column of the wave's first column
        constexpr float NEG = -__builtin_huge_valf();
        float mx = NEG;
        static_for<2>([&](auto J) {
          static_for<16>([&](auto R) {
            constexpr int j = J, r = R;
            const int c = cb + 32 * j + 8 * (r / 4) + 4 * lh + (r % 4);
            if (c < g.dN) mx = fmaxf(mx, acc[i][j][r]);
          });
        });
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        float sm = 0.0f;
        if (mx != NEG) {
          static_for<2>([&](auto J) {
            static_for<16>([&](auto R) {
              constexpr int j = J, r = R;
              const int c = cb + 32 * j + 8 * (r / 4) + 4 * lh + (r % 4);
              if (c < g.dN) sm += __expf(acc[i][j][r] - mx);
            });
          });
        }
        sm += __shfl_xor(sm, 32, 64);
        if (rok) {
          const int ng = (g.dN + 63) >> 6;
          if (lh == 0 && cb < g.dN)
            reinterpret_cast<float2*>(g.dc)[row * ng + (cb >> 6)] = make_float2(mx, sm);
          const int64_t tc = (int64_t)g.target[row] - g.v0 - cb;
          if (tc >= 0 && tc < 64 && cb + tc < g.dN && ((tc >> 2) & 1) == lh) {
            const int want = static_cast<int>(tc) & ~4;  // 32 j + 8 q + u
            float val = 0.0f;
            static_for<2>([&](auto J) {
              static_for<16>([&](auto R) {
                constexpr int j = J, r = R;
                // a sum of selects (one term matches): the compiler keeps
                // it in registers instead of indexing the accumulators
                val += 32 * j + 8 * (r / 4) + (r % 4) == want ? acc[i][j][r] : 0.0f;
              });
            });
            g.yt[row] = val;
          }
        }
      } else if constexpr (MODE == RT_DX || MODE == VOC_DX) {
        // fp32 outputs through the patch, 16 rows at a time ([16][64] fp32,
        // 256-byte rows, 16-byte chunk c of row r at c ^ r); each lane then
        // finishes 8 consecutive outputs of one row:
        //   RT_DX: dx = bf16([float(dx) +] v)   (one rounding)
        //   VOC_DX: dxa[b] = v (first block) or dxa[b] + v
        const int cg = lane & 7;
        const int col = n0 + wn * 64 + 8 * cg;
        static_for<2>([&](auto H) {
          constexpr int h = H;
          if ((l32 >> 4) == h) {
            const int rr = l32 & 15;
            static_for<2>([&](auto J) {
              static_for<4>([&](auto Q) {
                constexpr int j = J, q = Q;
                const int c = 8 * j + 2 * q + lh;
                put16(rr * 256 + ((c ^ rr) << 4),
                      make_float4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                  acc[i][j][4 * q + 3]));
              });
            });
          }
          fence();
          static_for<2>([&](auto Tt) {
            constexpr int t = Tt;
            const int rr = 8 * t + (lane >> 3);
            const float4 d0 = getf16(rr * 256 + (((2 * cg) ^ rr) << 4));
            const float4 d1 = getf16(rr * 256 + (((2 * cg + 1) ^ rr) << 4));
            const int rt = rb + 16 * h + rr;
            if (rt < mvalid && col < g.dN) {
              const int64_t row = (int64_t)m0 + rt;
              float v[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
              if constexpr (MODE == RT_DX) {
                uint4* o = reinterpret_cast<uint4*>(static_cast<uint16_t*>(g.dc) + row * g.c_ld + col);
                if (g.flag) {
                  const uint4 u = *o;
                  const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
                  for (int q = 0; q < 4; ++q) {
                    v[2 * q] = bf16_lo(w4[q]) + v[2 * q];
                    v[2 * q + 1] = bf16_hi(w4[q]) + v[2 * q + 1];
                  }
                }
                *o = make_uint4(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7]));
              } else {
                float4* o = reinterpret_cast<float4*>(static_cast<float*>(g.dc) +
                                                      (int64_t)e * g.c_bstride + row * g.c_ld + col);
                if (!g.flag) {
                  const float4 a = o[0], b = o[1];
                  v[0] += a.x; v[1] += a.y; v[2] += a.z; v[3] += a.w;
                  v[4] += b.x; v[5] += b.y; v[6] += b.z; v[7] += b.w;
                }
                o[0] = make_float4(v[0], v[1], v[2], v[3]);
                o[1] = make_float4(v[4], v[5], v[6], v[7]);
              }
            }
          });
          fence();
        });
      } else {
        // one bf16 output, [32][64] bf16, 128-byte rows, 16-byte chunk c of
        // row r at c ^ ((r / 2) % 8)
        if constexpr (MODE == VOC_GRAD) {
          // the logit gradient of each value, G = dl ([v == t] - exp(y - lse)),
          // 0 past the block's columns
          const int rt = rb + l32;
          float lse = 0.0f, dl = 0.0f;
          int64_t tc = -1;
          if (rt < mvalid) {
            const int64_t row = (int64_t)m0 + rt;
            lse = g.lse[row];
            dl = g.dloss[row];
            tc = (int64_t)g.target[row] - g.v0;
          }
          static_for<2>([&](auto J) {
            static_for<16>([&](auto R) {
              constexpr int j = J, r = R;
              const int c = n0 + wn * 64 + 32 * j + 8 * (r / 4) + 4 * lh + (r % 4);
              const float p = __expf(acc[i][j][r] - lse);
              acc[i][j][r] = c < g.dN ? dl * ((c == tc ? 1.0f : 0.0f) - p) : 0.0f;
            });
          });
        }
        static_for<2>([&](auto J) {
          static_for<4>([&](auto Q) {
            constexpr int j = J, q = Q;
            const int off = l32 * 128 + (((4 * j + q) ^ ((l32 >> 1) & 7)) << 4) + ((lh ^ (l32 >> 4)) & 1) * 8;
            put8(off, pack4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]));
          });
        });
        fence();
        static_for<4>([&](auto Tt) {
          constexpr int t = Tt;
          const int r = 8 * t + (lane >> 3), c = lane & 7;
          const uint4 v = unswap(get16(r * 128 + ((c ^ ((r >> 1) & 7)) << 4)), r);
          const int rt = rb + r, col = n0 + wn * 64 + 8 * c;
          // column limit: d; the block's columns (VOC_DW); G's whole pitch,
          // zeros past the block included (VOC_GRAD)
          const int climit = MODE == VOC_GRAD ? static_cast<int>(g.c_ld) : DENSE ? g.dN : d;
          if (rt < mvalid && col < climit) {
            uint16_t* out;
            if constexpr (MODE == FWD_DOWN) out = g.y + (int64_t)(seg + m0 + rt) * d;
            else if constexpr (MODE == DGRAD_GATE_UP) out = g.dx + (int64_t)(seg + m0 + rt) * d;
            else if constexpr (MODE == WGRAD_DOWN) out = g.dwd + e * wdf + (int64_t)(m0 + rt) * d;
            else if constexpr (MODE == VOC_GRAD) out = static_cast<uint16_t*>(g.dc) + (int64_t)(m0 + rt) * g.c_ld;
            else out = static_cast<uint16_t*>(g.dc) + (int64_t)(m0 + rt) * g.c_ld + g.cc0;  // VOC_DW
            *reinterpret_cast<uint4*>(out + col) = v;
          }
        });
        fence();
      }
    });
  };

  // zero weight-gradient tile (expert without rows)
  auto zero_tile = [&](const Tile& tl) __attribute__((always_inline)) {
    const int R = (MODE == WGRAD_GATE_UP) ? d : f;   // output rows
    const int C = (MODE == WGRAD_GATE_UP) ? f : d;   // output columns
    const int cw = DUAL ? BN / 2 : BN;               // tile columns per output
    const int nout = DUAL ? 2 : 1;
    for (int idx = threadIdx.x; idx < BM * (cw / 8) * nout; idx += NTHR) {
      const int o = idx / (BM * (cw / 8));
      const int rem = idx % (BM * (cw / 8));
      const int r = tl.m0 + rem / (cw / 8), c = tl.n0 + (rem % (cw / 8)) * 8;
      if (r < R && c < C) {
        uint16_t* base = (MODE == WGRAD_GATE_UP) ? (o ? g.dwu : g.dwg) : g.dwd;
        *reinterpret_cast<uint4*>(base + tl.e * wdf + (int64_t)r * C + c) = make_uint4(0u, 0u, 0u, 0u);
      }
    }
  };

  const Tables tb{g.mt_start, g.offsets, g.wk_start, g.nz_start};
  // Schedule choice (uniform over the launch).  The weight gradients
  // (grouped, and the vocabulary's dW) read both operands with transposing
  // LDS reads; when their tiles are long (at least 16 K steps on average)
  // they run the ping-pong schedule below, which keeps those reads out of
  // the MFMA stream.  Its tile change costs five extra phases, so short
  // tiles, the router's dW (short token chunks) and every other mode run the
  // single-barrier schedule after it.
  constexpr bool PP_OK = WGRAD || MODE == VOC_DW;
  bool use_pp = false;
  if constexpr (PP_OK) {
    if constexpr (DENSE) use_pp = g.kspan >= 16 * BK;
    else use_pp = 16 * tb.nz(g.E_loc) <= tb.wk(g.E_loc);
  }
  if (use_pp) {
    if constexpr (PP_OK) {
      // ---------------------------------------------------------- LDS ring
      // NA = 2 slots of UNIT bytes for operand A (loaded one step ahead), then
      // 3 for operand B (two steps ahead).  Both operands are N-contiguous.
      constexpr int NA = 2;
      using St = NStream<4>;
      static_assert(A_N && !B_K && NRING - NA == 3 && 2 * St::LH == 8,
                    "the wait counts below assume this ring and 8 loads per wave and step");
      lds_char* const ring = (lds_char*)(lds);  // address-space cast
      const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));
      struct Frags {
        bf16x8 a[4], b[2];
      };
      // fragments of sub-step `sub` (16 k, 0..3) of the step held in A's ring
      // slot `sa` and B's ring slot `sb`
      auto load_frags = [&](Frags& F, int sa, int sb, int sub) __attribute__((always_inline)) {
        const lds_char* ta = ring + sa * UNIT + (sub >> 1) * HALF;
        const lds_char* tbl = ring + (NA + sb) * UNIT + (sub >> 1) * HALF;
#pragma unroll
        for (int i = 0; i < 4; ++i) F.a[i] = AOp::frag(ta, arow[i], sub & 1, lane);
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) F.b[jj] = BOp::frag(tbl, brow[jj], sub & 1, lane);
      };
      // the 8 MFMAs of one sub-step, kept in this order and apart from any
      // other instruction
      auto mma = [&](const Frags& F) __attribute__((always_inline)) {
        static_for<8>([&](auto T) {
          constexpr int t = T;
          acc[t / 2][t % 2] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.b[t % 2], F.a[t / 2], acc[t / 2][t % 2], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
        });
      };
      // End of a phase: this wave's LDS reads are done, then the workgroup
      // barrier.  One asm statement, so the compiler moves no memory access
      // across it.
      auto phase_end = []() __attribute__((always_inline)) {
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);
      };

      // ------------------------------------------------------ write-out
      // A finished tile leaves in four passes, one per 32-row block i of
      // every wave's 128 x 64 accumulator block: each wave writes its block i
      // as bf16 into its 4 KiB patch of a pass slot (wave X at X * 4 KiB),
      // and after the barrier the four waves of group 1 each store a quarter
      // of the pass as 256-byte row pieces.  The patch layouts carry XOR
      // swizzles that keep the 64 banks conflict-free (bf16 rows 16..31 hold
      // their two 8-byte halves swapped).
      typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
      typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
      auto unswap = [](uint4 v, int r) __attribute__((always_inline)) {
        return (r & 16) ? make_uint4(v.z, v.w, v.x, v.y) : v;
      };
      auto put_block = [&](auto IC, lds_char* patch) __attribute__((always_inline)) {
        constexpr int i = IC;
        const int ln = opaque(threadIdx.x & 63);
        const int p32 = ln & 31, ph = ln >> 5;
        auto put8 = [&](int off, uint2 v) __attribute__((always_inline)) {
          *(__attribute__((address_space(3))) u32x2v*)(patch + off) = u32x2v{v.x, v.y};
        };
        if constexpr (DUAL) {
          // gate [32][32] bf16 at +0, up at +2048; 64-byte rows, 16-byte
          // chunk c of row r at c ^ ((r / 4) % 4)
          static_for<4>([&](auto Q) {
            constexpr int q = Q;
            const int off = p32 * 64 + ((q ^ ((p32 >> 2) & 3)) << 4) + ((ph ^ (p32 >> 4)) & 1) * 8;
            put8(off, pack4(acc[i][0][4 * q], acc[i][0][4 * q + 1], acc[i][0][4 * q + 2], acc[i][0][4 * q + 3]));
            put8(2048 + off, pack4(acc[i][1][4 * q], acc[i][1][4 * q + 1], acc[i][1][4 * q + 2],
                                   acc[i][1][4 * q + 3]));
          });
        } else {
          // [32][64] bf16, 128-byte rows, 16-byte chunk c of row r at
          // c ^ ((r / 2) % 8)
          static_for<2>([&](auto J) {
            static_for<4>([&](auto Q) {
              constexpr int j = J, q = Q;
              const int off = p32 * 128 + (((4 * j + q) ^ ((p32 >> 1) & 7)) << 4) + ((ph ^ (p32 >> 4)) & 1) * 8;
              put8(off, pack4(acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]));
            });
          });
        }
      };
      // Pass i's rows (block i of every wave's accumulators, in slot S) to
      // memory, one quarter per wave q of group 1, as rows of 256 bytes:
      // dual, the row half wm = q % 2 of output q / 2 (gate, up) across the
      // four column groups; otherwise the row half wm and column groups
      // 2 (q / 2) and 2 (q / 2) + 1.  Each store instruction covers 4 rows;
      // each group of 16 lanes reads 256 consecutive patch bytes.
      auto store_pass = [&](const Tile& tl, auto IC, const lds_char* S) __attribute__((always_inline)) {
        constexpr int i = IC;
        const int e = tl.e, m0 = tl.m0, n0 = tl.n0;
        const int ln = opaque(threadIdx.x & 63);
        const int mvalid = DENSE ? (g.dM - m0) : ((MODE == WGRAD_GATE_UP ? d : f) - m0);
        const int qm = w & 1, qh = (w >> 1) & 1;  // this wave's quarter (group 1)
        const int rb = qm * 128 + 32 * i;  // tile row of the block's first row
        if (rb >= mvalid) return;
        auto get16 = [&](const lds_char* patch, int off) __attribute__((always_inline)) {
          const u32x4v v = *(const __attribute__((address_space(3))) u32x4v*)(patch + off);
          return make_uint4(v[0], v[1], v[2], v[3]);
        };
        if constexpr (DUAL) {
          const int xn = ln >> 4, rr = (ln >> 2) & 3, c = ln & 3;
          const lds_char* patch = S + (qm + 2 * xn) * PATCH_BYTES + qh * 2048;
          uint16_t* const out = (qh ? g.dwu : g.dwg) + e * wdf;
          const int col = n0 + xn * 32 + 8 * c;
          static_for<8>([&](auto Tt) {
            constexpr int t = Tt;
            const int r = 4 * t + rr;
            const uint4 v = unswap(get16(patch, r * 64 + ((c ^ (t & 3)) << 4)), r);
            const int rt = rb + r;
            if (rt < mvalid && col < f)
              *reinterpret_cast<uint4*>(out + (int64_t)(m0 + rt) * f + col) = v;
          });
        } else {
          const int xn = 2 * qh + (ln >> 5), rr = (ln >> 3) & 3, c = ln & 7;
          const lds_char* patch = S + (qm + 2 * xn) * PATCH_BYTES;
          const int col = n0 + xn * 64 + 8 * c;
          static_for<8>([&](auto Tt) {
            constexpr int t = Tt;
            const int r = 4 * t + rr;
            const uint4 v = unswap(get16(patch, r * 128 + ((c ^ ((r >> 1) & 7)) << 4)), r);
            const int rt = rb + r;
            if (rt < mvalid && col < (DENSE ? g.dN : d)) {
              uint16_t* o;
              if constexpr (MODE == WGRAD_DOWN) o = g.dwd + e * wdf + (int64_t)(m0 + rt) * d;
              else o = static_cast<uint16_t*>(g.dc) + (int64_t)(m0 + rt) * g.c_ld + g.cc0;  // VOC_DW
              *reinterpret_cast<uint4*>(o + col) = v;
            }
          });
        }
      };

      // -------------------------------------------------------- tile stream
      // Waves 0-3 (group 0, one per SIMD) and waves 4-7 (group 1) each hold
      // half of the tile's B-side columns.  Time runs in phases separated by
      // workgroup barriers: in a memory phase a group reads the fragments of
      // one half step (two sub-steps) from LDS, in the compute phase that
      // follows it runs that half step's 16 MFMAs per wave and nothing else;
      // group 1 runs one phase behind group 0, so on every SIMD one wave
      // issues MFMAs while the other moves data.
      //   The roles are split: group 0 issues every operand load and never
      // stores, group 1 issues every output store and never waits for vector
      // memory.  A wave's vector-memory counter completes in issue order, so
      // a wave that stored a tile and then waits for the next tile's operands
      // would wait for its stores too.  Group 0 loads A step j + 1 in its
      // first memory phase of step j and B up to step j + 2 in its second
      // (a B step that lay beyond the next tile when its turn came, after a
      // tile of one step, goes out here too), and waits for A and B step
      // j + 1 at the end of step j.  Loads for steps past the current tile
      // fetch the next tile's first steps (its streams are prepared before
      // the tile's last two steps).
      //   Between tiles, group 0 first waits out group 1's last half step;
      // then four write-out passes run in the two slots the finished tile's
      // last step used (A's and B's), group 1 storing pass p - 1 while every
      // wave writes pass p.  Group 0's first memory phase of the new tile
      // runs beside group 1's store of the last pass; A step 1 and B step 2
      // of the new tile go to those two slots after it.  Every wave passes
      // the same number of barriers: two per half step, five per tile
      // change, and one more at the start (group 1: the stagger) or at a
      // tile change with no tile after it (group 0).
      const int grp = w >> 2, wq = w & 3;
      auto run = [&](auto GC) __attribute__((always_inline)) {
        constexpr int G = GC;
        TileIter<MODE> it;
        it.init(g, tb);
        Tile tc = it.next(g, tb);
        if (!tc.valid) return;
        St ca, cb, na, nb;  // group 0: A and B loads of the current and of the next tile
        auto prep = [&](const Tile& t, St& sa, St& sb) __attribute__((always_inline)) {
          AOp oa;
          setupA(t, oa);
          sa.setup(oa, wq, lane);
          BOp ob;
          setupB(t, ob);
          sb.setup(ob, wq, lane);
        };
        // one step of one operand into LDS unit `u` (its two halves)
        auto issue = [&](const St& st, int j, uint32_t u) __attribute__((always_inline)) {
          st.issue(j, 0, u, wq);
          st.issue(j, 1, u + HALF, wq);
        };
        zero_acc();
        int ra = 0, rb = 0;  // ring slots (A: 0..1, B: 0..2) of the current step
        int bl = 0;          // group 0: first B step, counted in the current tile, not yet issued
        if constexpr (G == 0) {
          // prologue: A step 0, B steps 0 and 1 (of this tile)
          prep(tc, ca, cb);
          issue(ca, 0, lds0);
          for (bl = 0; bl < 2 && bl < tc.nk; ++bl) issue(cb, bl, lds0 + (NA + bl) * UNIT);
        }
        wait_vmcnt<0>();
        phase_end();
        if constexpr (G == 1) phase_end();

        Frags F0, F1;
        Tile tp;  // the tile written out at the start of the next one
        bool has_prev = false;
        while (true) {
          if (has_prev) {
            // write-out passes in the finished tile's last-step slots
            lds_char* const S0 = ring + (ra ^ 1) * UNIT;
            lds_char* const S1 = ring + (NA + (rb == 0 ? 2 : rb - 1)) * UNIT;
            if constexpr (G == 0) phase_end();
            lgkm_drained();
            static_for<4>([&](auto P) {
              constexpr int p = P;
              put_block(P, (p & 1 ? S1 : S0) + w * PATCH_BYTES);
              if constexpr (G == 1 && p > 0)
                store_pass(tp, std::integral_constant<int, p - 1>{}, (p - 1) & 1 ? S1 : S0);
              phase_end();
            });
            zero_acc();
            if constexpr (G == 1) {
              store_pass(tp, std::integral_constant<int, 3>{}, S1);
              if (tc.valid) phase_end();
            }
          }
          if (!tc.valid) break;
          const int nk = tc.nk;
          int nkn = 0;  // group 0: steps of the next tile (0: none)
          // step j counted in the current tile (past nk: the next tile's) of
          // operand A or B into LDS unit `u`; false if its tile is neither
          // the current nor the next one
          auto issue_at = [&](bool b_side, int j, uint32_t u) __attribute__((always_inline)) {
            if (j < nk) {
              issue(b_side ? cb : ca, j, u);
              return true;
            }
            if (j - nk < nkn) {
              issue(b_side ? nb : na, j - nk, u);
              return true;
            }
            return false;
          };
          // One K step: two half steps, each a memory and a compute phase.
          // TAIL: its loads may reach past the tile (the next one or nothing).
          auto step = [&](int s, auto TAILC) __attribute__((always_inline)) {
            constexpr bool TAIL = TAILC;
            // ---- memory phase, first half (group 0: A step s + 1)
            if constexpr (G == 0) {
              const uint32_t u = lds0 + (ra ^ 1) * UNIT;
              if constexpr (TAIL) issue_at(false, s + 1, u);
              else issue(ca, s + 1, u);
            }
            lgkm_drained();
            load_frags(F0, ra, rb, 0);
            load_frags(F1, ra, rb, 1);
            phase_end();
            // ---- compute phase, first half
            mma(F0);
            mma(F1);
            phase_end();
            // ---- memory phase, second half (group 0: B up to step s + 2)
            bool b8 = false;  // group 0: B step s + 2 went out this step, the last of its loads
            if constexpr (G == 0) {
              while (bl <= s + 2) {
                const int d3 = rb + bl - s;  // 1 or 2: B steps s and earlier are in place
                const uint32_t u = lds0 + (NA + (d3 >= 3 ? d3 - 3 : d3)) * UNIT;
                if constexpr (TAIL) {
                  if (!issue_at(true, bl, u)) break;
                } else {
                  issue(cb, bl, u);
                }
                ++bl;
              }
              b8 = bl == s + 3;
            }
            load_frags(F0, ra, rb, 2);
            load_frags(F1, ra, rb, 3);
            phase_end();
            // ---- compute phase, second half; group 0 then waits for A and B
            // step s + 1 (B step s + 2, issued after them, may still fly)
            mma(F0);
            mma(F1);
            if constexpr (G == 0) {
              if (b8) wait_vmcnt<8>();
              else wait_vmcnt<0>();
            }
            phase_end();
            ra ^= 1;
            rb = rb == 2 ? 0 : rb + 1;
          };
          int s = 0;
          for (; s + 2 < nk; ++s) step(s, std::false_type{});
          // the last two steps load into the next tile: prepare its streams
          const Tile tn = it.next(g, tb);
          if constexpr (G == 0) {
            if (tn.valid) {
              prep(tn, na, nb);
              nkn = tn.nk;
            }
          }
          for (; s < nk; ++s) step(s, std::true_type{});
          tp = tc;
          has_prev = true;
          tc = tn;
          if constexpr (G == 0) {
            ca = na;
            cb = nb;
            bl -= nk;
          }
        }
        wait_vmcnt<0>();
      };
      if (grp == 0) run(std::integral_constant<int, 0>{});
      else run(std::integral_constant<int, 1>{});
    }
  } else {
    // ------------------------------------------------------------ LDS rings
    // NA = 2 slots of UNIT bytes for operand A, then NB = 3 for operand B, one
    // K step per slot.  A (called F below) is loaded one step ahead, B (S) two:
    // in the forward and data-gradient GEMMs B is the expert weights, whose
    // tiles miss L2 more often; in the weight gradients B is dH (the reverse
    // order measured 5 % slower there).  The single sync of step s (after its
    // last fragment reads) waits for step s + 1, then prepares F for step s + 2
    // and S for step s + 3, into the slots step s has freed (an N-contiguous
    // operand as two halves of 32 k).  These loads go out between the eight
    // MFMAs that follow the sync, F's first, so the matrix cores have work
    // while they are issued and the issue state is never held across
    // sub-steps (holding it across the whole step costs scalar-register
    // spills and a branch per load).
    constexpr bool A_K = !A_N, B_N = !B_K;
    constexpr int NA = 2, NB = NRING - NA;
    constexpr int LA = A_K ? KStream<false, NWAVE>::LK : 2 * NStream<NWAVE>::LH;  // loads per wave of one step's issue
    constexpr int LB = B_K ? KStream<false, NWAVE>::LK : 2 * NStream<NWAVE>::LH;
    // At the sync of step s the loads issued after the last of F(s + 1) (the
    // later of the two operands it needs) are S(s + 2)'s four: the
    // vector-memory count it may leave.
    constexpr int X_END = 4;
    static_assert(!(A_N && B_K), "no mode has an N-contiguous A with a K-contiguous B");
    static_assert(LA == 4 && LB == 4 && NA == 2 && NB == 3,
                  "the sync count assumes this ring");

    lds_char* const ring = (lds_char*)(lds);  // address-space cast
    const uint32_t lds0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(ring));
    struct Frags {
      bf16x8 a[4], b[2];
    };
    // fragments of sub-step `sub` (16 k, 0..3) of the step held in A's ring
    // slot `sa` and B's ring slot `sb`
    auto load_frags = [&](Frags& F, int sa, int sb, int sub) __attribute__((always_inline)) {
      const lds_char* ta = ring + sa * UNIT + (A_N ? (sub >> 1) * HALF : 0);
      const lds_char* tb = ring + (NA + sb) * UNIT + (B_N ? (sub >> 1) * HALF : 0);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (A_N) F.a[i] = AOp::frag(ta, arow[i], sub & 1, lane);
        else F.a[i] = AOp::frag(ta, arow[i] + l32, sub, lh);
      }
#pragma unroll
      for (int jj = 0; jj < 2; ++jj) {
        if constexpr (B_K) F.b[jj] = BOp::frag(tb, brow[jj] + l32, sub, lh);
        else F.b[jj] = BOp::frag(tb, brow[jj], sub & 1, lane);
      }
    };
    // one fragment f of sub-step `sub` (f = 0..3: A's row blocks, 4..5: B's)
    auto load_frag1 = [&](Frags& F, int sa, int sb, int sub, auto FI) __attribute__((always_inline)) {
      constexpr int f = FI;
      if constexpr (f < 4) {
        const lds_char* ta = ring + sa * UNIT + (A_N ? (sub >> 1) * HALF : 0);
        if constexpr (A_N) F.a[f] = AOp::frag(ta, arow[f], sub & 1, lane);
        else F.a[f] = AOp::frag(ta, arow[f] + l32, sub, lh);
      } else {
        const lds_char* tb = ring + (NA + sb) * UNIT + (B_N ? (sub >> 1) * HALF : 0);
        if constexpr (B_K) F.b[f - 4] = BOp::frag(tb, brow[f - 4] + l32, sub, lh);
        else F.b[f - 4] = BOp::frag(tb, brow[f - 4], sub & 1, lane);
      }
    };
    auto mma = [&](const Frags& F) __attribute__((always_inline)) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int jj = 0; jj < 2; ++jj)
          acc[i][jj] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.b[jj], F.a[i], acc[i][jj], 0, 0, 0);
    };

    // ---------------------------------------------------------- tile stream
    // Tiles run one after another, each with its own K loop; A is loaded one
    // step and B two steps ahead of the sync that needs them.  Near a tile's
    // end those loads fetch the next tile's first steps (its load streams are
    // prepared when the current tile starts).  A load that would reach still
    // further (the next tile has fewer steps than the look-ahead) is issued
    // out of range into its slot, so every sync's count stays exact, and is
    // issued again for real when its tile starts, after a full wait.  After a
    // tile's last step, B's slot of that step holds the epilogue patches; its
    // refill waits for the epilogue.
    using AStream = typename std::conditional<A_N, NStream<NWAVE>, KStream<MODE == DGRAD_GATE_UP, NWAVE>>::type;
    using BStream = typename std::conditional<B_N, NStream<NWAVE>, KStream<MODE == DGRAD_GATE_UP, NWAVE>>::type;
    const i32x4 nil = make_rsrc(nullptr, 0);
    TileIter<MODE> it;
    it.init(g, tb);
    zero_acc();
    Tile tc = it.next(g, tb);
    if (tc.valid) {
      AStream sa, xa;  // loads of this tile and of the next one
      BStream sb, xb;
      auto prep = [&](const Tile& t, AStream& a, BStream& b) __attribute__((always_inline)) {
        AOp ao;
        setupA(t, ao);
        a.setup(ao, w, lane);
        BOp bo;
        setupB(t, bo);
        b.setup(bo, w, lane);
      };
      // part p (0, 1) of one step's loads of an operand into ring slot `slot`:
      // the two halves of an N-contiguous step; a K-contiguous step at p = 0
      auto issA = [&](const AStream& st, int j, int slot, int p) __attribute__((always_inline)) {
        const uint32_t u = lds0 + slot * UNIT;
        if constexpr (A_N) st.issue(j, p, u + p * HALF, w);
        else if (p == 0) st.issue(j, u, w);
      };
      auto noneA = [&](int slot, int p) __attribute__((always_inline)) {
        const uint32_t u = lds0 + slot * UNIT;
        if constexpr (A_N) NStream<NWAVE>::none(nil, u + p * HALF, w);
        else if (p == 0) KStream<false, NWAVE>::none(nil, u, w);
      };
      auto issB = [&](const BStream& st, int j, int slot, int p) __attribute__((always_inline)) {
        const uint32_t u = lds0 + (NA + slot) * UNIT;
        if constexpr (B_N) st.issue(j, p, u + p * HALF, w);
        else if (p == 0) st.issue(j, u, w);
      };
      auto noneB = [&](int slot, int p) __attribute__((always_inline)) {
        const uint32_t u = lds0 + (NA + slot) * UNIT;
        if constexpr (B_N) NStream<NWAVE>::none(nil, u + p * HALF, w);
        else if (p == 0) KStream<false, NWAVE>::none(nil, u, w);
      };

      prep(tc, sa, sb);
      // prologue: the loads the syncs of steps -3, -2, -1 would have issued
      // (B 0; A 0, B 1; A 1, B 2), steps past the tile out of range
      {
        const int nk = tc.nk;
        auto pa = [&](int j) {
          static_for<2>([&](auto P) {
            if (j < nk) issA(sa, j, j, P); else noneA(j, P);
          });
        };
        auto pb = [&](int j) {
          static_for<2>([&](auto P) {
            if (j < nk) issB(sb, j, j, P); else noneB(j, P);
          });
        };
        pb(0);
        pa(0);
        pb(1);
        pa(1);
        pb(2);
      }
      wait_vmcnt<X_END>();
      lgkm_drained();
      __builtin_amdgcn_s_barrier();
      __builtin_amdgcn_sched_barrier(0);

      Frags cur, nxt;
      int ra = 0, rb = 0;  // ring slots (A: 0..1, B: 0..2) of the step being computed
      load_frags(cur, 0, 0, 0);
      auto sync = [&]() __attribute__((always_inline)) {
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");  // this wave's fragment reads are done
      };
      // the 8 MFMAs of one sub-step on F, with the six fragment reads of the
      // next sub-step (into G) between the first three, in the order the next
      // sub-step's MFMAs need them (a0 b0 | b1 a1 | a2 a3), so that each has
      // five or more MFMAs to arrive
      auto mma_read = [&](const Frags& F, Frags& G, int sa, int sb, int sub) __attribute__((always_inline)) {
        static_for<8>([&](auto T) {
          constexpr int t = T;
          acc[t / 2][t % 2] =
              __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.b[t % 2], F.a[t / 2], acc[t / 2][t % 2], 0, 0, 0);
          __builtin_amdgcn_sched_barrier(0);
          if constexpr (t < 6) {
            constexpr int f0 = t == 0 ? 0 : t == 1 ? 4 : t == 2 ? 5 : t == 3 ? 1 : t == 4 ? 2 : 3;
            load_frag1(G, sa, sb, sub, std::integral_constant<int, f0>{});
            __builtin_amdgcn_sched_barrier(0);
          }
        });
      };
      while (true) {
        const int nk = tc.nk;
        Tile tn;
        tn.valid = false;
        int nkn = 0;
        unsigned done_a = 0, done_b = 0;  // steps of the next tile loaded for real
        // part p of the A / B loads aimed at tile step j (past nk: the next tile)
        auto loadA = [&](int j, int slot, int p) __attribute__((always_inline)) {
          if (j < nk) {
            issA(sa, j, slot, p);
          } else if (j - nk < nkn) {
            issA(xa, j - nk, slot, p);
            done_a |= 1u << (j - nk);
          } else {
            noneA(slot, p);
          }
        };
        auto loadB = [&](int j, int slot, int p) __attribute__((always_inline)) {
          if (j < nk) {
            issB(sb, j, slot, p);
          } else if (j - nk < nkn) {
            issB(xb, j - nk, slot, p);
            done_b |= 1u << (j - nk);
          } else {
            noneB(slot, p);
          }
        };
        // One K step.  TAIL: its look-ahead loads may reach past the tile
        // (the next tile or nothing); otherwise they stay inside it.  LAST:
        // the tile's last step (B's refill waits for the epilogue).
        auto step = [&](int ks, auto TAIL, auto LAST) __attribute__((always_inline)) {
          constexpr bool tail = TAIL, last = LAST;
          const int ra1 = ra ^ 1, rb1 = rb == 2 ? 0 : rb + 1;  // slots of the next step
          mma_read(cur, nxt, ra, rb, 1);
          mma_read(nxt, cur, ra, rb, 2);
          mma_read(cur, nxt, ra, rb, 3);
          sync();
          wait_vmcnt<X_END>();
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
          // this step's slots are free: A's refill with step ks + 2, B's with
          // ks + 3 (deferred past the epilogue on the tile's last step)
          if constexpr (!last) {
            lgkm_drained();
            load_frags(cur, ra1, rb1, 0);
            __builtin_amdgcn_sched_barrier(0);
            // the 8 MFMAs of sub-step 3 with the loads between them (A's parts
            // after the second and fourth, B's after the sixth and eighth)
            static_for<8>([&](auto T) {
              constexpr int t = T;
              acc[t / 2][t % 2] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                  nxt.b[t % 2], nxt.a[t / 2], acc[t / 2][t % 2], 0, 0, 0);
              __builtin_amdgcn_sched_barrier(0);
              if constexpr (t % 2 == 1) {
                if constexpr (t < 4) {
                  if constexpr (tail) loadA(ks + 2, ra, t / 2);
                  else issA(sa, ks + 2, ra, t / 2);
                } else {
                  if constexpr (tail) loadB(ks + 3, rb, t / 2 - 2);
                  else issB(sb, ks + 3, rb, t / 2 - 2);
                }
                __builtin_amdgcn_sched_barrier(0);
              }
            });
            lgkm_drained();
          } else {
            loadA(ks + 2, ra, 0);
            loadA(ks + 2, ra, 1);
            __builtin_amdgcn_sched_barrier(0);
            mma(nxt);
          }
          __builtin_amdgcn_sched_barrier(0);
          ra = ra1;
          rb = rb1;
        };
        int ks = 0;
        // steps whose loads stay inside the tile
        for (; ks + NB < nk; ++ks) step(ks, std::false_type{}, std::false_type{});
        // the last steps reach into the next tile: prepare its loads now
        tn = it.next(g, tb);
        if (tn.valid) {
          prep(tn, xa, xb);
          nkn = tn.nk;
        }
        for (; ks + 1 < nk; ++ks) step(ks, std::true_type{}, std::false_type{});
        step(ks, std::true_type{}, std::true_type{});
        // epilogue patches: B's slot of the tile's last step
        const int rlast = rb == 0 ? 2 : rb - 1;
        lds_char* const patch = ring + (NA + rlast) * UNIT + w * PATCH_BYTES;
        epilogue(tc, patch);
        zero_acc();
        // the patch reads are done once the LDS counter drains; the stores stay
        // in flight.  The next sync's vector-memory wait covers them: the
        // operations it may leave in flight are B's refill loads below, issued
        // after them (stores and loads share that counter but need not
        // complete in order relative to each other, so a wait may only leave
        // loads in flight that were issued after everything it must cover).
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        __builtin_amdgcn_s_barrier();  // every wave is done with its patch
        __builtin_amdgcn_sched_barrier(0);
        if (!tn.valid) break;
        // B's deferred refill (tile step nk + 2 = the next tile's step 2)
        loadB(nk + 2, rlast, 0);
        loadB(nk + 2, rlast, 1);
        tc = tn;
        sa = xa;
        sb = xb;
        // Steps of the new tile that a shorter tile before it could not load
        // ahead went out as out-of-range loads: issue them now into their
        // slots and wait for every load (rare: only after tiles of fewer
        // steps than the look-ahead).
        const unsigned need_a = (1u << min(tc.nk, NA)) - 1u, need_b = (1u << min(tc.nk, NB)) - 1u;
        if ((done_a & need_a) != need_a || (done_b & need_b) != need_b) {
          for (int j = 0; j < min(tc.nk, NA); ++j)
            if (!((done_a >> j) & 1u)) {
              const int sl = (ra + j) & 1;
              issA(sa, j, sl, 0);
              issA(sa, j, sl, 1);
            }
          for (int j = 0; j < min(tc.nk, NB); ++j)
            if (!((done_b >> j) & 1u)) {
              const int sl = (rb + j) % 3;
              issB(sb, j, sl, 0);
              issB(sb, j, sl, 1);
            }
          wait_vmcnt<0>();
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
        }
        lgkm_drained();
        load_frags(cur, ra, rb, 0);
      }
      // the last steps' out-of-range loads still write their (zero) slots:
      // let them land before the workgroup's LDS is released
      wait_vmcnt<0>();
    }
  }
  if constexpr (WGRAD) {
    // experts without rows: their weight gradients are exact zeros
    TileIter<MODE> itz;
    itz.init(g, tb, true);
    for (Tile tz = itz.next(g, tb); tz.valid; tz = itz.next(g, tb)) zero_tile(tz);
  }
}

// Per-expert prefixes over experts in index order: row tiles (mt_start), K
// steps (wk_start) and experts with rows (nz_start).  One workgroup,
// E_loc <= 1024.
__global__ __launch_bounds__(1024) void gemm_sched_kernel(const int32_t* __restrict__ offsets,
                                                          int E_loc, int32_t* __restrict__ mt_start,
                                                          int32_t* __restrict__ wk_start,
                                                          int32_t* __restrict__ nz_start) {
  __shared__ int wsum[3][16];
  const int e = threadIdx.x;
  const int n = (e < E_loc) ? offsets[e + 1] - offsets[e] : 0;
  const int v[3] = {(n + BM - 1) / BM, (n + BK - 1) / BK, n > 0 ? 1 : 0};
  int32_t* const out[3] = {mt_start, wk_start, nz_start};
  const int lane = e & 63, w = e >> 6;
  int incl[3] = {v[0], v[1], v[2]};
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
#pragma unroll
    for (int c = 0; c < 3; ++c) {
      const int u = __shfl_up(incl[c], o, 64);
      if (lane >= o) incl[c] += u;
    }
  }
  if (lane == 63)
#pragma unroll
    for (int c = 0; c < 3; ++c) wsum[c][w] = incl[c];
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    int base = 0;
    for (int q = 0; q < w; ++q) base += wsum[c][q];
    if (e < E_loc) out[c][e] = base + incl[c] - v[c];
    if (e == E_loc - 1) out[c][E_loc] = base + incl[c];
  }
}

struct GemmWs {
  int32_t* mt_start;
  int32_t* wk_start;
  int32_t* nz_start;
  uint16_t* act;
  uint16_t* dhg;
  uint16_t* dhu;
};

GemmWs carve(void* ws, int64_t cap, int E_loc, int f, bool bwd) {
  char* p = static_cast<char*>(ws);
  GemmWs w{};
  w.mt_start = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (E_loc + 1), 256);
  w.wk_start = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (E_loc + 1), 256);
  w.nz_start = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (E_loc + 1), 256);
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
  grouped_gemm_kernel<MODE><<<static_cast<unsigned>(blocks), NTHR, 0, s>>>(a);
  prof_end(kid, s);
  return hipGetLastError();
}

// Persistent grid: one workgroup per CU (a multiple of the 8 XCDs).
int64_t pgrid() {
  const int64_t g = (device_cus() / NXCD) * NXCD;
  return g > 0 ? g : NXCD;
}

hipError_t sched(const int32_t* offsets, int E_loc, const GemmWs& w, hipStream_t s) {
  prof_begin(K_GEMM_SCHED, s);
  gemm_sched_kernel<<<1, 1024, 0, s>>>(offsets, E_loc, w.mt_start, w.wk_start, w.nz_start);
  prof_end(K_GEMM_SCHED, s);
  return hipGetLastError();
}

}  // namespace

size_t gemm_ws_bytes(int64_t cap, int E_loc, int d, int f, unsigned flags) {
  (void)d;
  const bool bwd = flags != 0;
  const size_t act_bytes = align_up(sizeof(uint16_t) * static_cast<size_t>(cap) * f, 256);
  return 3 * align_up(sizeof(int32_t) * (E_loc + 1), 256) + act_bytes * (bwd ? 3 : 1) + 256;
}

hipError_t launch_ffn_fwd(const uint16_t* x_perm, const int32_t* offsets, int E_loc, int64_t cap,
                          int d, int f, const uint16_t* wg, const uint16_t* wu,
                          const uint16_t* wd, uint16_t* hg, uint16_t* hu, uint16_t* y,
                          void* ws, hipStream_t s) {
  GemmWs w = carve(ws, cap, E_loc, f, false);
  if (hipError_t e = sched(offsets, E_loc, w, s); e != hipSuccess) return e;
  GemmArgs a{};
  a.x_perm = x_perm; a.wg = wg; a.wu = wu; a.wd = wd;
  a.offsets = offsets; a.mt_start = w.mt_start; a.wk_start = w.wk_start; a.nz_start = w.nz_start;
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
  a.offsets = offsets; a.mt_start = w.mt_start; a.wk_start = w.wk_start; a.nz_start = w.nz_start;
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

// ------------------------------------------------------ dense products
namespace {
template <int MODE>
hipError_t run_dense(GemmArgs& a, int kid, hipStream_t s) {
  a.MT = static_cast<int>(ceil_div(a.dM, BM));
  a.NT = static_cast<int>(ceil_div(a.dN, Traits<MODE>::DUAL ? BN / 2 : BN));
  if (a.MT <= 0 || a.NT <= 0 || a.batches <= 0) return hipSuccess;
  return run_gemm<MODE>(a, pgrid(), kid, s);
}
}  // namespace

hipError_t launch_router_dw_mfma(const uint16_t* x, const uint16_t* dl3, int64_t T, int d, int E,
                                 int64_t ld3, int64_t chunk, float* part, hipStream_t s) {
  GemmArgs a{};
  a.da = x; a.db = dl3; a.dc = part;
  a.a_ld = d; a.b_ld = ld3; a.c_ld = E; a.c_bstride = static_cast<int64_t>(d) * E;
  a.dM = d; a.dN = E; a.dK = static_cast<int>(T); a.dE = E;
  a.kspan = static_cast<int>(chunk); a.batches = static_cast<int>(ceil_div(T, chunk));
  return run_dense<RT_DW>(a, K_ROUTE_DW, s);
}

hipError_t launch_router_dx_mfma(const uint16_t* dl3, const uint16_t* w3, int64_t T, int d, int E,
                                 int64_t ld3, int accumulate, uint16_t* dx, hipStream_t s) {
  GemmArgs a{};
  a.da = dl3; a.db = w3; a.dc = dx;
  a.a_ld = ld3; a.b_ld = d; a.c_ld = d;
  a.dM = static_cast<int>(T); a.dN = d; a.dK = 3 * E; a.kspan = 3 * E; a.batches = 1;
  a.flag = accumulate;
  return run_dense<RT_DX>(a, K_ROUTE_DX, s);
}

hipError_t launch_vocab_logits_mfma(const uint16_t* x, const uint16_t* w, int64_t ldw, int64_t bc0,
                                    int64_t v0, int N, int H, int vb, const int32_t* target,
                                    float* part, float* yt, hipStream_t s) {
  GemmArgs a{};
  a.da = x; a.db = w; a.dc = part; a.target = target; a.yt = yt;
  a.a_ld = H; a.b_ld = ldw; a.bc0 = bc0; a.v0 = v0;
  a.dM = N; a.dN = vb; a.dK = H; a.kspan = H; a.batches = 1;
  return run_dense<VOC_FWD>(a, K_VOC_LOGITS, s);
}

hipError_t launch_vocab_grad_mfma(const uint16_t* x, const uint16_t* w, int64_t ldw, int64_t bc0,
                                  int64_t v0, int N, int H, int vb, const int32_t* target,
                                  const float* lse, const float* dloss, uint16_t* G, int64_t gp,
                                  hipStream_t s) {
  GemmArgs a{};
  a.da = x; a.db = w; a.dc = G; a.target = target; a.lse = lse; a.dloss = dloss;
  a.a_ld = H; a.b_ld = ldw; a.c_ld = gp; a.bc0 = bc0; a.v0 = v0;
  a.dM = N; a.dN = vb; a.dK = H; a.kspan = H; a.batches = 1;
  return run_dense<VOC_GRAD>(a, K_VOC_GRAD, s);
}

hipError_t launch_vocab_dx_mfma(const uint16_t* G, int64_t gp, const uint16_t* w, int64_t ldw,
                                int64_t bc0, int N, int H, int vb, int kspan, int first,
                                float* dxa, hipStream_t s) {
  GemmArgs a{};
  a.da = G; a.db = w; a.dc = dxa;
  a.a_ld = gp; a.b_ld = ldw; a.c_ld = H; a.c_bstride = static_cast<int64_t>(N) * H; a.bc0 = bc0;
  a.dM = N; a.dN = H; a.dK = vb; a.kspan = kspan;
  a.batches = static_cast<int>(ceil_div(vb, kspan));
  a.flag = first;
  return run_dense<VOC_DX>(a, K_VOC_DX, s);
}

hipError_t launch_vocab_dw_mfma(const uint16_t* x, const uint16_t* G, int64_t gp, int N, int H,
                                int vb, uint16_t* dw, int64_t ldd, int64_t cc0, hipStream_t s) {
  GemmArgs a{};
  a.da = x; a.db = G; a.dc = dw;
  a.a_ld = H; a.b_ld = gp; a.c_ld = ldd; a.cc0 = cc0;
  a.dM = H; a.dN = vb; a.dK = N; a.kspan = N; a.batches = 1;
  return run_dense<VOC_DW>(a, K_VOC_DW, s);
}

}  // namespace moe
