// Least-loaded expert parallelism on the device (Mixture-of-Parallelisms
// Sec. 3.3, recap of LLEP: each call measures the work every rank holds; a
// rank above its share hands part of it, with the weights of the experts
// concerned, to ranks below their share; the set of products computed stays
// the same).
//
// llep_plan_kernel: one workgroup turns the per-expert assignment counts
// into per-rank row windows of every expert.  Load is counted in units of g
// rows (g = 1: rows; g = the grouped GEMM's row-tile height: the tiles a
// rank's products run, as a window of w rows costs ceil(w / g) of them):
// each rank keeps its own experts (ascending) up to the capacity
// C = max(ceil(capacity / g), ceil(U / E_p)) units, U = sum ceil(n_e / g);
// the spill of every expert, largest first in units (ties: lower index),
// goes in pieces of whole units to whichever rank has the fewest units
// (ties: lower rank).  Expert e's assignments, in the layer's stable row
// order, are cut into consecutive windows: the home rank's first, then the
// pieces in the order handed out; every window but an expert's last is a
// whole number of units, so no window splits a tile.
//
// llep_window_kernel: one rank's share of an all-expert permutation: the
// rows of its windows, compacted per expert, and the dst map of the
// assignments it computes (every other assignment gets -1).  The rank then
// runs the grouped GEMMs over all E experts (a shipped expert's weights are
// read where they lie) and a partial combine.
#include "common.h"

namespace moe {
namespace {

constexpr int PT = 1024;  // threads of the plan and offsets kernels

__global__ __launch_bounds__(PT) void llep_plan_kernel(const int32_t* __restrict__ counts, int E,
                                                       int E_p, int capacity, int g,
                                                       int32_t* __restrict__ lo,
                                                       int32_t* __restrict__ hi,
                                                       int32_t* __restrict__ load_out,
                                                       int32_t* __restrict__ n_ship_out) {
  __shared__ int n_s[MOE_MAX_E];
  __shared__ int spill_s[MOE_MAX_E];
  __shared__ uint64_t key_s[MOE_MAX_E];
  __shared__ int load_s[64];   // units
  __shared__ int rows_s[64];   // rows
  __shared__ int wsum[PT / 64];
  const int tid = threadIdx.x;
  const int G = E / E_p;

  // total units and the capacity (in units)
  int v = 0;
  for (int e = tid; e < E; e += PT) {
    n_s[e] = counts[e];
    v += (counts[e] + g - 1) / g;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  if ((tid & 63) == 0) wsum[tid >> 6] = v;
  for (int64_t q = tid; q < static_cast<int64_t>(E_p) * E; q += PT) {
    lo[q] = 0;
    hi[q] = 0;
  }
  __syncthreads();
  int total = 0;
#pragma unroll
  for (int w = 0; w < PT / 64; ++w) total += wsum[w];
  const int C = max(capacity / g + (capacity % g != 0), (total + E_p - 1) / E_p);

  // keep at home: rank r walks its G experts in ascending order
  if (tid < E_p) {
    int ld = 0, rows = 0;
    for (int e = tid * G; e < (tid + 1) * G; ++e) {
      const int u = (n_s[e] + g - 1) / g;
      const int keep = min(u, C - ld);
      const int keep_rows = static_cast<int>(min<int64_t>(n_s[e], static_cast<int64_t>(keep) * g));
      hi[static_cast<int64_t>(tid) * E + e] = keep_rows;
      ld += keep;
      rows += keep_rows;
      spill_s[e] = u - keep;
    }
    load_s[tid] = ld;
    rows_s[tid] = rows;
  }
  __syncthreads();

  // order the spilled experts: spill descending, index ascending; experts
  // without spill sort last.  Bitonic sort of the next power of two >= E.
  int P2 = 1;
  while (P2 < E) P2 <<= 1;
  for (int e = tid; e < P2; e += PT)
    key_s[e] = (e < E && spill_s[e] > 0)
                   ? (static_cast<uint64_t>(0x7fffffff - spill_s[e]) << 32) | static_cast<uint32_t>(e)
                   : ~0ull;
  __syncthreads();
  for (int size = 2; size <= P2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = tid; i < P2; i += PT) {
        const int j = i ^ stride;
        if (j > i) {
          const bool up = (i & size) == 0;
          const uint64_t a = key_s[i], b = key_s[j];
          if ((a > b) == up) {
            key_s[i] = b;
            key_s[j] = a;
          }
        }
      }
      __syncthreads();
    }
  }

  // hand out the spill, one wave: lane r holds rank r's load (units, rows)
  if (tid < 64) {
    const int lane = tid;
    int ld = lane < E_p ? load_s[lane] : 0x7fffffff;
    int rows = lane < E_p ? rows_s[lane] : 0;
    int ships = 0;
    // every piece but the last of an expert fills a rank, so there are at
    // most E + E_p pieces: the bound ends the loop even on inconsistent input
    int budget = E + E_p;
    for (int q = 0; q < E && budget > 0; ++q) {
      const uint64_t key = key_s[q];
      if (key == ~0ull) break;
      const int e = static_cast<int>(key & 0xffffffffu);
      int left = 0x7fffffff - static_cast<int>(key >> 32);  // spilled units
      int s = static_cast<int>(static_cast<int64_t>((n_s[e] + g - 1) / g - left) * g);  // first spilled row
      while (left > 0 && budget-- > 0) {
        // least loaded rank, lower rank on ties
        uint64_t best = (static_cast<uint64_t>(static_cast<uint32_t>(ld)) << 32) | static_cast<uint32_t>(lane);
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) {
          const uint64_t other = __shfl_xor(best, o, 64);
          best = other < best ? other : best;
        }
        const int r = static_cast<int>(best & 0xffffffffu);
        const int room = C - static_cast<int>(best >> 32);
        const int take = min(left, room);
        if (take <= 0) break;  // no room anywhere: capacity below the total
        const int nr = static_cast<int>(min<int64_t>(n_s[e] - s, static_cast<int64_t>(take) * g));
        if (lane == 0) {
          lo[static_cast<int64_t>(r) * E + e] = s;
          hi[static_cast<int64_t>(r) * E + e] = s + nr;
        }
        if (lane == r) {
          ld += take;
          rows += nr;
        }
        s += nr;
        left -= take;
        ++ships;
      }
    }
    if (lane < E_p) load_out[lane] = rows;
    if (lane == 0) *n_ship_out = ships;
  }
}

// offsets_r = exclusive scan of this rank's window sizes (E <= 1024),
// clamped to the row capacity: rows past it are never addressed
__global__ __launch_bounds__(PT) void llep_offsets_kernel(const int32_t* __restrict__ lo,
                                                          const int32_t* __restrict__ hi, int E,
                                                          int64_t cap,
                                                          int32_t* __restrict__ offsets_r) {
  __shared__ int wsum[PT / 64];
  const int e = threadIdx.x;
  const int v = e < E ? hi[e] - lo[e] : 0;
  const int lane = e & 63, w = e >> 6;
  int incl = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int u = __shfl_up(incl, o, 64);
    if (lane >= o) incl += u;
  }
  if (lane == 63) wsum[w] = incl;
  __syncthreads();
  int before = 0;
  for (int q = 0; q < w; ++q) before += wsum[q];
  if (e < E) offsets_r[e] = static_cast<int32_t>(min<int64_t>(before + incl - v, cap));
  if (e == E - 1) offsets_r[E] = static_cast<int32_t>(min<int64_t>(before + incl, cap));
}

// per assignment a: its row on this rank (or -1), and the inverse map
__global__ __launch_bounds__(256) void llep_window_kernel(
    const int32_t* __restrict__ idx, const int32_t* __restrict__ offsets_all,
    const int32_t* __restrict__ dst_all, const int32_t* __restrict__ lo,
    const int32_t* __restrict__ hi, const int32_t* __restrict__ offsets_r, int64_t A, int E,
    int32_t* __restrict__ row_src_r, int32_t* __restrict__ dst_r) {
  const int64_t a = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
  if (a >= A) return;
  const int e = idx[a];
  int q = -1;
  // an expert id outside [0, E) (caller garbage) or an assignment missing
  // from the permutation is computed by no rank
  if (static_cast<unsigned>(e) >= static_cast<unsigned>(E) || dst_all[a] < 0) {
    dst_r[a] = -1;
    return;
  }
  const int g = dst_all[a] - offsets_all[e];  // position among expert e's assignments
  if (g >= lo[e] && g < hi[e]) {
    q = offsets_r[e] + (g - lo[e]);
    if (q < offsets_r[e + 1]) row_src_r[q] = static_cast<int32_t>(a);
    else q = -1;  // past the row capacity (an inconsistent plan)
  }
  dst_r[a] = q;
}

}  // namespace

hipError_t launch_llep_plan(const int32_t* counts, int E, int E_p, int capacity, int granule,
                            int32_t* lo, int32_t* hi, int32_t* load, int32_t* n_ship, hipStream_t s) {
  prof_begin(K_LLEP_PLAN, s);
  llep_plan_kernel<<<1, PT, 0, s>>>(counts, E, E_p, capacity, granule, lo, hi, load, n_ship);
  prof_end(K_LLEP_PLAN, s);
  return hipGetLastError();
}

hipError_t launch_llep_dispatch(const uint16_t* x, const int32_t* idx, const int32_t* offsets_all,
                                const int32_t* dst_all, const int32_t* lo, const int32_t* hi,
                                int64_t T, int d, int E, int k, int64_t cap, int32_t* offsets_r,
                                int32_t* row_src_r, int32_t* dst_r, uint16_t* x_perm_r,
                                hipStream_t s) {
  prof_begin(K_LLEP_WINDOW, s);
  llep_offsets_kernel<<<1, PT, 0, s>>>(lo, hi, E, cap, offsets_r);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  const int64_t A = T * k;
  if (A > 0)
    llep_window_kernel<<<static_cast<unsigned>(ceil_div(A, 256)), 256, 0, s>>>(
        idx, offsets_all, dst_all, lo, hi, offsets_r, A, E, row_src_r, dst_r);
  prof_end(K_LLEP_WINDOW, s);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  if (A == 0) return hipSuccess;
  return launch_gather(x, dst_r, T, d, k, x_perm_r, s);
}

}  // namespace moe
