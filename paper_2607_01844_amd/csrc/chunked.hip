// Memory-efficient forward of the expert layer: the permute -> grouped
// SwiGLU -> combine pipeline over chunks of tokens, alternating between two
// streams with two sets of transient buffers.  Only two chunks' routed rows,
// expert intermediates and expert outputs are resident at any instant
// instead of all T*k of them (the O(N k H + N_r I) activation peak of the
// layer), and one chunk's permutation and combine (HBM-bound) overlap the
// other chunk's grouped GEMMs.  Every output row depends only on its own
// token, so the result is bit-identical to the unchunked forward.
//
// The expert-range variant forms the whole layer's permutation index once
// and walks the permuted rows in chunks of consecutive rows (consecutive
// experts, the first and last possibly in part): each chunk's rows are
// gathered, multiplied, and written into one y_perm of all rows, and one
// combine forms y.  An expert's weights are then read by the one or two
// chunks its rows fall in, where token chunks read every expert's weights
// once per chunk; the transient is y_perm plus two chunks' rows,
// intermediates and activations.  Every y_perm row depends only on its own
// token and expert and the combine is the unchunked one, so y is again
// bit-identical to the unchunked forward.
//
// Host code only: the kernels are the ones of route/permute/gemm/combine.
#include <mutex>

#include "common.h"

namespace moe {
namespace {

struct ChunkSet {
  int32_t* offsets;  // [E_loc + 1]
  int32_t* row_src;  // [cap_c]
  int32_t* dst;      // [chunk * k]
  uint16_t* x_perm;  // [cap_c][d]
  uint16_t* h_gate;  // [cap_c][f]
  uint16_t* h_up;    // [cap_c][f]
  uint16_t* y_perm;  // [cap_c][d]
  void* perm_ws;
  void* gemm_ws;
};

size_t set_bytes(int64_t chunk, int E, int k, int E_loc, int d, int f) {
  const int64_t cap = chunk * std::min(k, E_loc);
  size_t b = 0;
  b += align_up(sizeof(int32_t) * (E_loc + 1), 256);
  b += align_up(sizeof(int32_t) * static_cast<size_t>(cap), 256);
  b += align_up(sizeof(int32_t) * static_cast<size_t>(chunk) * k, 256);
  b += 2 * align_up(sizeof(uint16_t) * static_cast<size_t>(cap) * d, 256);
  b += 2 * align_up(sizeof(uint16_t) * static_cast<size_t>(cap) * f, 256);
  b += align_up(permute_ws_bytes(chunk, E, k, E_loc), 256);
  b += align_up(gemm_ws_bytes(cap, E_loc, d, f, 0), 256);
  return b;
}

ChunkSet carve_set(char*& p, int64_t chunk, int E, int k, int E_loc, int d, int f) {
  const int64_t cap = chunk * std::min(k, E_loc);
  ChunkSet c;
  auto take = [&p](size_t bytes) {
    char* q = p;
    p += align_up(bytes, 256);
    return q;
  };
  c.offsets = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (E_loc + 1)));
  c.row_src = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * static_cast<size_t>(cap)));
  c.dst = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * static_cast<size_t>(chunk) * k));
  c.x_perm = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(cap) * d));
  c.y_perm = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(cap) * d));
  c.h_gate = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(cap) * f));
  c.h_up = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(cap) * f));
  c.perm_ws = take(permute_ws_bytes(chunk, E, k, E_loc));
  c.gemm_ws = take(gemm_ws_bytes(cap, E_loc, d, f, 0));
  return c;
}

// `to` waits for everything queued on `from` so far.  One event per device,
// created on first use and kept for the life of the process; the record and
// the wait happen under one lock, so concurrent calls cannot cross them.
constexpr int kMaxDev = 64;
hipError_t stream_after(hipStream_t to, hipStream_t from) {
  static std::mutex mu;
  static hipEvent_t ev[kMaxDev] = {};
  int dev = 0;
  if (hipError_t e = hipGetDevice(&dev); e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDev) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> g(mu);
  if (ev[dev] == nullptr) {
    if (hipError_t e = hipEventCreateWithFlags(&ev[dev], hipEventDisableTiming); e != hipSuccess)
      return e;
  }
  if (hipError_t e = hipEventRecord(ev[dev], from); e != hipSuccess) return e;
  return hipStreamWaitEvent(to, ev[dev], 0);
}

}  // namespace

size_t ffn_fwd_chunked_ws_bytes(int64_t chunk, int E, int k, int E_loc, int d, int f) {
  return 2 * set_bytes(chunk, E, k, E_loc, d, f) + 256;
}

hipError_t launch_ffn_fwd_chunked(const uint16_t* x, const int32_t* idx, const float* gate,
                                  int64_t T, int d, int E, int k, int e_begin, int E_loc, int f,
                                  const uint16_t* wg, const uint16_t* wu, const uint16_t* wd,
                                  int64_t chunk, uint16_t* y, void* ws, hipStream_t s0,
                                  hipStream_t s1) {
  if (T == 0) return hipSuccess;
  char* p = static_cast<char*>(ws);
  ChunkSet set[2] = {carve_set(p, chunk, E, k, E_loc, d, f), carve_set(p, chunk, E, k, E_loc, d, f)};
  const bool two = s1 != s0;
  if (two) {  // stream 1 starts after everything the caller queued on stream 0
    if (hipError_t e = stream_after(s1, s0); e != hipSuccess) return e;
  }
  const int64_t nchunks = ceil_div(T, chunk);
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t t0 = c * chunk, tc = std::min(chunk, T - t0);
    const int64_t cap = tc * std::min(k, E_loc);
    ChunkSet& b = set[c & 1];
    hipStream_t st = (two && (c & 1)) ? s1 : s0;
    // a buffer set is reused by chunks c and c + 2 on the same stream: in order
    if (hipError_t e = launch_permute(x + t0 * d, idx + t0 * k, tc, d, E, k, e_begin, E_loc,
                                      b.offsets, nullptr, b.row_src, b.dst, b.x_perm, b.perm_ws,
                                      st);
        e != hipSuccess)
      return e;
    if (hipError_t e = launch_ffn_fwd(b.x_perm, b.offsets, E_loc, cap, d, f, wg, wu, wd, b.h_gate,
                                      b.h_up, b.y_perm, b.gemm_ws, st);
        e != hipSuccess)
      return e;
    if (hipError_t e = launch_combine(b.y_perm, b.dst, gate + t0 * k, tc, d, k, y + t0 * d, st);
        e != hipSuccess)
      return e;
  }
  if (two) {  // the call's work is complete on stream 0 once stream 1's part is
    if (hipError_t e = stream_after(s0, s1); e != hipSuccess) return e;
  }
  return hipSuccess;
}


namespace {

struct RowSet {
  int32_t* offsets;  // [E_loc + 1], relative to the chunk's first row
  uint16_t* x_perm;  // [rc][d]
  uint16_t* h_gate;  // [rc][f]
  uint16_t* h_up;    // [rc][f]
  void* gemm_ws;
};

struct RowLayout {
  int64_t cap, rc;
  size_t index_bytes, set_bytes;
};

RowLayout row_layout(int64_t T, int E, int k, int E_loc, int d, int f, int64_t chunk_rows) {
  RowLayout L;
  L.cap = T * std::min(k, E_loc);
  L.rc = std::max<int64_t>(1, std::min(chunk_rows, L.cap));
  // the whole layer's offsets, row_src, dst, the permutation's workspace and y_perm
  L.index_bytes = align_up(sizeof(int32_t) * (E_loc + 1), 256) +
                  align_up(sizeof(int32_t) * static_cast<size_t>(L.cap), 256) +
                  align_up(sizeof(int32_t) * static_cast<size_t>(T) * k, 256) +
                  align_up(permute_ws_bytes(T, E, k, E_loc), 256) +
                  align_up(sizeof(uint16_t) * static_cast<size_t>(L.cap) * d, 256);
  L.set_bytes = align_up(sizeof(int32_t) * (E_loc + 1), 256) +
                align_up(sizeof(uint16_t) * static_cast<size_t>(L.rc) * d, 256) +
                2 * align_up(sizeof(uint16_t) * static_cast<size_t>(L.rc) * f, 256) +
                align_up(gemm_ws_bytes(L.rc, E_loc, d, f, 0), 256);
  return L;
}

}  // namespace

size_t ffn_fwd_row_chunked_ws_bytes(int64_t T, int E, int k, int E_loc, int d, int f,
                                    int64_t chunk_rows) {
  const RowLayout L = row_layout(T, E, k, E_loc, d, f, chunk_rows);
  return L.index_bytes + 2 * L.set_bytes + 256;
}

hipError_t launch_ffn_fwd_row_chunked(const uint16_t* x, const int32_t* idx, const float* gate,
                                      int64_t T, int d, int E, int k, int e_begin, int E_loc,
                                      int f, const uint16_t* wg, const uint16_t* wu,
                                      const uint16_t* wd, int64_t chunk_rows, uint16_t* y,
                                      void* ws, hipStream_t s0, hipStream_t s1) {
  if (T == 0) return hipSuccess;
  const RowLayout L = row_layout(T, E, k, E_loc, d, f, chunk_rows);
  char* p = static_cast<char*>(ws);
  auto take = [&p](size_t bytes) {
    char* q = p;
    p += align_up(bytes, 256);
    return q;
  };
  int32_t* offsets = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (E_loc + 1)));
  int32_t* row_src = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * static_cast<size_t>(L.cap)));
  int32_t* dst = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * static_cast<size_t>(T) * k));
  void* perm_ws = take(permute_ws_bytes(T, E, k, E_loc));
  uint16_t* y_perm = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(L.cap) * d));
  RowSet set[2];
  for (RowSet& b : set) {
    b.offsets = reinterpret_cast<int32_t*>(take(sizeof(int32_t) * (E_loc + 1)));
    b.x_perm = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(L.rc) * d));
    b.h_gate = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(L.rc) * f));
    b.h_up = reinterpret_cast<uint16_t*>(take(sizeof(uint16_t) * static_cast<size_t>(L.rc) * f));
    b.gemm_ws = take(gemm_ws_bytes(L.rc, E_loc, d, f, 0));
  }
  // the whole layer's index (offsets, row_src, dst), without gathering rows
  if (hipError_t e = launch_permute(x, idx, T, d, E, k, e_begin, E_loc, offsets, nullptr, row_src,
                                    dst, nullptr, perm_ws, s0);
      e != hipSuccess)
    return e;
  const bool two = s1 != s0;
  if (two) {  // stream 1 starts after the index (and the caller's work on stream 0)
    if (hipError_t e = stream_after(s1, s0); e != hipSuccess) return e;
  }
  const int64_t nchunks = ceil_div(L.cap, L.rc);
  for (int64_t c = 0; c < nchunks; ++c) {
    const int64_t r0 = c * L.rc, rc = std::min(L.rc, L.cap - r0);
    RowSet& b = set[c & 1];
    hipStream_t st = (two && (c & 1)) ? s1 : s0;
    // a buffer set is reused by chunks c and c + 2 on the same stream: in order
    if (hipError_t e = launch_chunk_rows(x, row_src, offsets, E_loc, r0, rc, d, k, b.offsets,
                                         b.x_perm, st);
        e != hipSuccess)
      return e;
    if (hipError_t e = launch_ffn_fwd(b.x_perm, b.offsets, E_loc, rc, d, f, wg, wu, wd, b.h_gate,
                                      b.h_up, y_perm + r0 * d, b.gemm_ws, st);
        e != hipSuccess)
      return e;
  }
  if (two) {  // every chunk's rows are in y_perm once stream 1's part is done
    if (hipError_t e = stream_after(s0, s1); e != hipSuccess) return e;
  }
  return launch_combine(y_perm, dst, gate, T, d, k, y, s0);
}

}  // namespace moe
