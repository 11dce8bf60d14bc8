// MoE expert-layer oracle: plain, slow, obviously-correct CPU reference.
//
// TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
// benchmark's CPU-baseline leg load this file's library.  It shares no code,
// header, table or helper with the HIP library, and it never calls it.
//
// What it computes is the plain MoE feed-forward layer of Mixture-of-
// Parallelisms (Sec. 2.1 "Mixture-of-Experts": a light router sends each
// token to its top-k of E experts; Sec. 3.1 notation H = d, I = f, N = T,
// eq. (peaks): N k H routed activations and N_r I expert intermediates).
// The paper's expert-parallel machinery (Sec. 3.3, LLEP and its memory-
// efficient variant) is lossless: it moves where each token-expert product is
// computed, never which experts a token uses or the result, so the plain
// layer below is the reference semantics for every placement of the work.
//
// Readings where the paper is silent (each one is also listed in the design
// notes of the repository):
//   R1 logits: fp32 fused-multiply-add chain over the hidden index j
//      ascending, starting from +0.0f, then one fp32 add of the bias.
//   R2 selection: the k largest logits by the total order (logit descending,
//      expert index ascending); -0.0 and +0.0 compare equal (a tie).
//   R3 slot order: slots 0..k-1 of a token follow that same order.
//   R4 gates: renorm = 0 -> softmax over all E logits evaluated at the chosen
//      experts; renorm = 1 -> softmax over the k chosen logits only.
//   R5 bias: added to the logits before both selection and softmax.
//   R6 rows of an expert segment are in ascending assignment order a = t*k+i
//      (a stable counting sort by local expert id).
//   R7 dropless: every local assignment is processed, no capacity limit.
//   R8 expert FFN: SwiGLU, silu(z) = z / (1 + exp(-z)),
//      Hg = X Wg, Hu = X Wu, A = silu(Hg) * Hu, O = A Wd.
//   R9 weight gradients overwrite (no accumulation); an expert with no rows
//      gets exactly zero gradients.
//
// Precision: template parameter In is the storage type of the inputs
// (uint16_t = bf16 bits, widened exactly; or double), R the arithmetic type
// (float or double).  Nothing is rounded to bf16 inside the oracle.
//
// Build: g++ -O2 -std=c++17 -fopenmp -mavx2 -mfma -ffp-contract=off -shared
// -fPIC (no -ffast-math: every sum below runs in the order written).

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <limits>
#include <vector>

namespace {

// ---------------------------------------------------------------- widening
inline float bf16_bits_to_float(uint16_t b) {
  uint32_t u = static_cast<uint32_t>(b) << 16;
  float f;
  std::memcpy(&f, &u, sizeof f);
  return f;
}
template <typename R> inline R widen(uint16_t b) { return static_cast<R>(bf16_bits_to_float(b)); }
template <typename R> inline R widen(double v) { return static_cast<R>(v); }
template <typename R> inline R widen(float v) { return static_cast<R>(v); }

template <typename R> inline R sigmoid(R z) { return R(1) / (R(1) + std::exp(-z)); }
// silu(z) = z * sigmoid(z)
template <typename R> inline R silu(R z) { return z * sigmoid(z); }
// d/dz silu(z) = s + z s (1 - s), s = sigmoid(z)
template <typename R> inline R silu_grad(R z) {
  R s = sigmoid(z);
  return s + z * s * (R(1) - s);
}

// ------------------------------------------------------------------ router
// R1 (fp32): logit[t][e] = fma chain over j ascending from +0.0f, then +bias.
template <typename In>
void logits_f32(const In* x, const float* w_r, const float* bias, int64_t T, int d, int E,
                float* logits) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    for (int e = 0; e < E; ++e) {
      float acc = +0.0f;
      for (int j = 0; j < d; ++j)
        acc = std::fma(widen<float>(x[t * d + j]), w_r[(int64_t)j * E + e], acc);
      if (bias) acc = acc + bias[e];
      logits[t * E + e] = acc;
    }
  }
}

// fp64 logits (for finite differences and the fp64 cross-check).
template <typename In, typename W>
void logits_f64(const In* x, const W* w_r, const W* bias, int64_t T, int d, int E,
                double* logits) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    for (int e = 0; e < E; ++e) {
      double acc = 0.0;
      for (int j = 0; j < d; ++j)
        acc += widen<double>(x[t * d + j]) * static_cast<double>(w_r[(int64_t)j * E + e]);
      if (bias) acc += static_cast<double>(bias[e]);
      logits[t * E + e] = acc;
    }
  }
}

// R2-R4: selection and gates from given logits.  Gate arithmetic is fp64
// (the method fixes no precision for the exponentials); G is the output type.
template <typename L, typename G>
void topk_gates(const L* logits, int64_t T, int E, int k, int renorm, int32_t* idx, G* gate) {
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    const L* l = logits + t * E;
    std::vector<int> order(E);
    std::iota(order.begin(), order.end(), 0);
    // total order: larger logit first; equal logits (including -0 == +0)
    // keep ascending expert index (stable sort of an ascending sequence); a
    // NaN logit ranks as -inf
    auto key = [&](int e) {
      return std::isnan(l[e]) ? -std::numeric_limits<L>::infinity() : l[e];
    };
    std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return key(a) > key(b); });
    const double m = static_cast<double>(l[order[0]]);
    double den = 0.0;
    if (renorm == 0) {
      for (int e = 0; e < E; ++e) den += std::exp(static_cast<double>(l[e]) - m);
    } else {
      for (int i = 0; i < k; ++i) den += std::exp(static_cast<double>(l[order[i]]) - m);
    }
    for (int i = 0; i < k; ++i) {
      idx[t * k + i] = order[i];
      gate[t * k + i] = static_cast<G>(std::exp(static_cast<double>(l[order[i]]) - m) / den);
    }
  }
}

// --------------------------------------------------------------- permutation
// Histogram, exclusive scan, and stable positions (R6).
void permute_index(const int32_t* idx, int64_t T, int E, int k, int e_begin, int E_loc,
                   int32_t* offsets, int32_t* counts_global, int32_t* row_src, int32_t* dst) {
  const int64_t A = T * k;
  std::vector<int64_t> cnt(E_loc, 0);
  if (counts_global)
    for (int e = 0; e < E; ++e) counts_global[e] = 0;
  for (int64_t a = 0; a < A; ++a) {
    const int e = idx[a];
    if (counts_global) counts_global[e] += 1;
    if (e >= e_begin && e < e_begin + E_loc) cnt[e - e_begin] += 1;
  }
  offsets[0] = 0;
  for (int e = 0; e < E_loc; ++e) offsets[e + 1] = static_cast<int32_t>(offsets[e] + cnt[e]);
  std::vector<int64_t> run(E_loc, 0);
  for (int64_t a = 0; a < A; ++a) {
    const int e = idx[a];
    if (e >= e_begin && e < e_begin + E_loc) {
      const int el = e - e_begin;
      const int64_t p = offsets[el] + run[el]++;
      row_src[p] = static_cast<int32_t>(a);
      dst[a] = static_cast<int32_t>(p);
    } else {
      dst[a] = -1;
    }
  }
}

// ------------------------------------------------------------- expert FFN
// One row through expert e (R8).  x: [d]; wg, wu: [d][f]; wd: [f][d].
template <typename In, typename R>
void ffn_fwd_row(const In* x, const In* wg, const In* wu, const In* wd, int d, int f,
                 R* hg, R* hu, R* a, R* y) {
  for (int n = 0; n < f; ++n) { hg[n] = R(0); hu[n] = R(0); }
  for (int j = 0; j < d; ++j) {
    const R xj = widen<R>(x[j]);
    const In* g = wg + (int64_t)j * f;
    const In* u = wu + (int64_t)j * f;
    for (int n = 0; n < f; ++n) {
      hg[n] += xj * widen<R>(g[n]);
      hu[n] += xj * widen<R>(u[n]);
    }
  }
  for (int n = 0; n < f; ++n) a[n] = silu(hg[n]) * hu[n];
  for (int c = 0; c < d; ++c) y[c] = R(0);
  for (int n = 0; n < f; ++n) {
    const R an = a[n];
    const In* w = wd + (int64_t)n * d;
    for (int c = 0; c < d; ++c) y[c] += an * widen<R>(w[c]);
  }
}

// Backward of one row given its upstream gradient dO = dy_row:
// dA = dO Wd^T; dHg = dA * Hu * silu'(Hg); dHu = dA * silu(Hg);
// dX = dHg Wg^T + dHu Wu^T.
template <typename In, typename R>
void ffn_bwd_row(const R* dy_row, const R* hg, const R* hu, const In* wg, const In* wu,
                 const In* wd, int d, int f, R* dhg, R* dhu, R* dx) {
  for (int n = 0; n < f; ++n) {
    const In* w = wd + (int64_t)n * d;
    R s = R(0);
    for (int c = 0; c < d; ++c) s += dy_row[c] * widen<R>(w[c]);
    dhg[n] = s * hu[n] * silu_grad(hg[n]);
    dhu[n] = s * silu(hg[n]);
  }
  for (int j = 0; j < d; ++j) {
    const In* g = wg + (int64_t)j * f;
    const In* u = wu + (int64_t)j * f;
    R s = R(0);
    for (int n = 0; n < f; ++n) s += dhg[n] * widen<R>(g[n]);
    for (int n = 0; n < f; ++n) s += dhu[n] * widen<R>(u[n]);
    dx[j] = s;
  }
}

}  // namespace

// ======================================================================
// exported entry points
// ======================================================================
extern "C" {

int oracle_abi_version(void) { return 1; }

// ---- router ---------------------------------------------------------------
void oracle_logits_f32_bf16(const uint16_t* x, const float* w_r, const float* bias, int64_t T,
                            int d, int E, float* logits) {
  logits_f32(x, w_r, bias, T, d, E, logits);
}
void oracle_logits_f64_bf16(const uint16_t* x, const float* w_r, const float* bias, int64_t T,
                            int d, int E, double* logits) {
  logits_f64(x, w_r, bias, T, d, E, logits);
}
void oracle_logits_f64_f64(const double* x, const double* w_r, const double* bias, int64_t T,
                           int d, int E, double* logits) {
  logits_f64(x, w_r, bias, T, d, E, logits);
}
void oracle_topk_f32(const float* logits, int64_t T, int E, int k, int renorm, int32_t* idx,
                     float* gate) {
  topk_gates(logits, T, E, k, renorm, idx, gate);
}
void oracle_topk_f64(const double* logits, int64_t T, int E, int k, int renorm, int32_t* idx,
                     double* gate) {
  topk_gates(logits, T, E, k, renorm, idx, gate);
}

// ---- permutation -----------------------------------------------------------
void oracle_permute_index(const int32_t* idx, int64_t T, int E, int k, int e_begin, int E_loc,
                          int32_t* offsets, int32_t* counts_global, int32_t* row_src,
                          int32_t* dst) {
  permute_index(idx, T, E, k, e_begin, E_loc, offsets, counts_global, row_src, dst);
}
// x_perm[p] = x[row_src[p] / k] (a copy of bf16 bits), p < M.
void oracle_gather_bf16(const uint16_t* x, const int32_t* row_src, int64_t M, int d, int k,
                        uint16_t* x_perm) {
#pragma omp parallel for schedule(static)
  for (int64_t p = 0; p < M; ++p) {
    const int64_t t = row_src[p] / k;
    std::memcpy(x_perm + p * d, x + t * d, sizeof(uint16_t) * d);
  }
}

// ---- expert FFN over explicit rows -----------------------------------------
// rows: n input rows x_rows[n][d]; expert[r] selects the (local) expert of row
// r in the stacked weights wg, wu [E_loc][d][f], wd [E_loc][f][d].
#define ORACLE_FFN_FWD(NAME, In, R)                                                        \
  void NAME(const In* x_rows, const int32_t* expert, int64_t n, int d, int f, const In* wg, \
            const In* wu, const In* wd, R* hg, R* hu, R* a, R* y) {                        \
    const int64_t wdf = (int64_t)d * f;                                                    \
    _Pragma("omp parallel for schedule(dynamic, 4)") for (int64_t r = 0; r < n; ++r) {     \
      const int64_t e = expert[r];                                                         \
      ffn_fwd_row<In, R>(x_rows + r * d, wg + e * wdf, wu + e * wdf, wd + e * wdf, d, f,   \
                         hg + r * f, hu + r * f, a + r * f, y + r * d);                    \
    }                                                                                      \
  }
ORACLE_FFN_FWD(oracle_ffn_fwd_rows_f32_bf16, uint16_t, float)
ORACLE_FFN_FWD(oracle_ffn_fwd_rows_f64_bf16, uint16_t, double)
ORACLE_FFN_FWD(oracle_ffn_fwd_rows_f64_f64, double, double)

#define ORACLE_FFN_BWD(NAME, In, R)                                                         \
  void NAME(const R* dy_rows, const R* hg, const R* hu, const int32_t* expert, int64_t n,  \
            int d, int f, const In* wg, const In* wu, const In* wd, R* dhg, R* dhu,        \
            R* dx_rows) {                                                                  \
    const int64_t wdf = (int64_t)d * f;                                                    \
    _Pragma("omp parallel for schedule(dynamic, 4)") for (int64_t r = 0; r < n; ++r) {     \
      const int64_t e = expert[r];                                                         \
      ffn_bwd_row<In, R>(dy_rows + r * d, hg + r * f, hu + r * f, wg + e * wdf,            \
                         wu + e * wdf, wd + e * wdf, d, f, dhg + r * f, dhu + r * f,       \
                         dx_rows + r * d);                                                 \
    }                                                                                      \
  }
ORACLE_FFN_BWD(oracle_ffn_bwd_rows_f32_bf16, uint16_t, float)
ORACLE_FFN_BWD(oracle_ffn_bwd_rows_f64_bf16, uint16_t, double)
ORACLE_FFN_BWD(oracle_ffn_bwd_rows_f64_f64, double, double)

// ---- weight gradients of one expert ----------------------------------------
// Rows 0..n-1 are the rows of that expert: X [n][d] (In), A, dHg, dHu [n][f]
// (R), dO [n][d] (R).  dWg[j][m] = sum_p X[p][j] dHg[p][m] (p ascending), etc.
// n = 0 gives exact zeros (R9).
#define ORACLE_WGRAD(NAME, In, R)                                                        \
  void NAME(const In* x_rows, const R* a, const R* dhg, const R* dhu, const R* dout,     \
            int64_t n, int d, int f, R* dwg, R* dwu, R* dwd) {                           \
    _Pragma("omp parallel for schedule(static)") for (int j = 0; j < d; ++j) {           \
      R* g = dwg + (int64_t)j * f;                                                       \
      R* u = dwu + (int64_t)j * f;                                                       \
      for (int m = 0; m < f; ++m) { g[m] = R(0); u[m] = R(0); }                          \
      for (int64_t p = 0; p < n; ++p) {                                                  \
        const R xj = widen<R>(x_rows[p * d + j]);                                        \
        for (int m = 0; m < f; ++m) {                                                    \
          g[m] += xj * dhg[p * f + m];                                                   \
          u[m] += xj * dhu[p * f + m];                                                   \
        }                                                                                \
      }                                                                                  \
    }                                                                                    \
    _Pragma("omp parallel for schedule(static)") for (int m = 0; m < f; ++m) {           \
      R* w = dwd + (int64_t)m * d;                                                       \
      for (int c = 0; c < d; ++c) w[c] = R(0);                                           \
      for (int64_t p = 0; p < n; ++p) {                                                  \
        const R am = a[p * f + m];                                                       \
        for (int c = 0; c < d; ++c) w[c] += am * dout[p * d + c];                        \
      }                                                                                  \
    }                                                                                    \
  }
ORACLE_WGRAD(oracle_wgrad_f32_bf16, uint16_t, float)
ORACLE_WGRAD(oracle_wgrad_f64_bf16, uint16_t, double)
ORACLE_WGRAD(oracle_wgrad_f64_f64, double, double)

// Selected entries of one expert's weight gradients, for large experts.
// which[s] = 0 (dWg[i][j]), 1 (dWu[i][j]) or 2 (dWd[i][j]); every entry is the
// same sum as above, with the needed columns of Hg, Hu, dA recomputed.
#define ORACLE_WGRAD_ENTRIES(NAME, In, R)                                                 \
  void NAME(const In* x_rows, const R* dout, int64_t n, int d, int f, const In* wg,       \
            const In* wu, const In* wd, const int32_t* which, const int32_t* ii,          \
            const int32_t* jj, int64_t ns, R* out) {                                      \
    _Pragma("omp parallel for schedule(dynamic, 1)") for (int64_t s = 0; s < ns; ++s) {   \
      const int m = (which[s] == 2) ? ii[s] : jj[s]; /* intermediate column */            \
      R acc = R(0);                                                                       \
      for (int64_t p = 0; p < n; ++p) {                                                   \
        R hgm = R(0), hum = R(0);                                                         \
        for (int j = 0; j < d; ++j) {                                                     \
          const R xj = widen<R>(x_rows[p * d + j]);                                       \
          hgm += xj * widen<R>(wg[(int64_t)j * f + m]);                                   \
          hum += xj * widen<R>(wu[(int64_t)j * f + m]);                                   \
        }                                                                                 \
        if (which[s] == 2) {                                                              \
          acc += silu(hgm) * hum * dout[p * d + jj[s]];                                   \
        } else {                                                                          \
          R da = R(0);                                                                    \
          for (int c = 0; c < d; ++c) da += dout[p * d + c] * widen<R>(wd[(int64_t)m * d + c]); \
          const R dh = (which[s] == 0) ? da * hum * silu_grad(hgm) : da * silu(hgm);      \
          acc += widen<R>(x_rows[p * d + ii[s]]) * dh;                                    \
        }                                                                                 \
      }                                                                                   \
      out[s] = acc;                                                                       \
    }                                                                                     \
  }
ORACLE_WGRAD_ENTRIES(oracle_wgrad_entries_f32_bf16, uint16_t, float)
ORACLE_WGRAD_ENTRIES(oracle_wgrad_entries_f64_bf16, uint16_t, double)

// ---- combine and its backward ----------------------------------------------
// out[t] = sum over slots i ascending with dst >= 0 of gate[t][i] * y[dst];
// gate == NULL means weight 1 (this is also the permutation's backward).
#define ORACLE_COMBINE(NAME, G, R)                                                        \
  void NAME(const R* y, const int32_t* dst, const G* gate, int64_t T, int d, int k,       \
            R* out) {                                                                     \
    _Pragma("omp parallel for schedule(static)") for (int64_t t = 0; t < T; ++t) {        \
      R* o = out + t * d;                                                                 \
      for (int c = 0; c < d; ++c) o[c] = R(0);                                            \
      for (int i = 0; i < k; ++i) {                                                       \
        const int64_t p = dst[t * k + i];                                                 \
        if (p < 0) continue;                                                              \
        const R g = gate ? static_cast<R>(gate[t * k + i]) : R(1);                        \
        for (int c = 0; c < d; ++c) o[c] += g * y[p * d + c];                             \
      }                                                                                   \
    }                                                                                     \
  }
ORACLE_COMBINE(oracle_combine_f32, float, float)
ORACLE_COMBINE(oracle_combine_f64, double, double)

// dy_perm[dst[t,i]] = gate[t,i] * dout[t];  dgate[t,i] = <dout[t], y[dst[t,i]]>
// (0 for a non-local slot).  dout arrives as In.
#define ORACLE_COMBINE_BWD(NAME, In, G, R)                                                \
  void NAME(const In* dout, const R* y, const int32_t* dst, const G* gate, int64_t T,     \
            int d, int k, R* dy_perm, R* dgate) {                                         \
    _Pragma("omp parallel for schedule(static)") for (int64_t t = 0; t < T; ++t) {        \
      for (int i = 0; i < k; ++i) {                                                       \
        const int64_t p = dst[t * k + i];                                                 \
        if (p < 0) {                                                                      \
          if (dgate) dgate[t * k + i] = R(0);                                             \
          continue;                                                                       \
        }                                                                                 \
        const R g = gate ? static_cast<R>(gate[t * k + i]) : R(1);                        \
        R s = R(0);                                                                       \
        for (int c = 0; c < d; ++c) {                                                     \
          const R dv = widen<R>(dout[t * d + c]);                                         \
          dy_perm[p * d + c] = g * dv;                                                    \
          s += dv * y[p * d + c];                                                         \
        }                                                                                 \
        if (dgate) dgate[t * k + i] = s;                                                  \
      }                                                                                   \
    }                                                                                     \
  }
ORACLE_COMBINE_BWD(oracle_combine_bwd_f32_bf16, uint16_t, float, float)
ORACLE_COMBINE_BWD(oracle_combine_bwd_f64_bf16, uint16_t, double, double)
ORACLE_COMBINE_BWD(oracle_combine_bwd_f64_f64, double, double, double)

// ---- router backward (fp64) ------------------------------------------------
// From dgate to d logits (softmax Jacobian at the chosen slots), then
// dW_r = x^T dlogits and dx_router = dlogits W_r^T.  The bias gradient is
// sum_t dlogits[t] (returned when dbias != NULL).
void oracle_router_dlogits_f64(const double* logits, const int32_t* idx, const double* gate,
                               const double* dgate, int64_t T, int E, int k, int renorm,
                               double* dl) {
  for (int64_t i = 0; i < T * E; ++i) dl[i] = 0.0;
  for (int64_t t = 0; t < T; ++t) {
    double* g = dl + t * E;
    if (renorm == 0) {
      // gate_i = p[e_i], p = softmax(l):  dl_e = sum_i dgate_i p_{e_i} (delta - p_e)
      double m = logits[t * E];
      for (int e = 1; e < E; ++e) m = std::max(m, logits[t * E + e]);
      double den = 0.0;
      for (int e = 0; e < E; ++e) den += std::exp(logits[t * E + e] - m);
      double s = 0.0;
      for (int i = 0; i < k; ++i) s += dgate[t * k + i] * gate[t * k + i];
      for (int e = 0; e < E; ++e) g[e] = -(std::exp(logits[t * E + e] - m) / den) * s;
      for (int i = 0; i < k; ++i) g[idx[t * k + i]] += dgate[t * k + i] * gate[t * k + i];
    } else {
      // gate_i = softmax over the chosen logits: dl_{e_i} = g_i (dgate_i - sum_j dgate_j g_j)
      double s = 0.0;
      for (int i = 0; i < k; ++i) s += dgate[t * k + i] * gate[t * k + i];
      for (int i = 0; i < k; ++i) g[idx[t * k + i]] = gate[t * k + i] * (dgate[t * k + i] - s);
    }
  }
}

void oracle_router_bwd_f64(const double* x, const double* w_r, const double* logits,
                           const int32_t* idx, const double* gate, const double* dgate,
                           int64_t T, int d, int E, int k, int renorm, double* dw_r,
                           double* dx, double* dbias) {
  std::vector<double> dl(static_cast<size_t>(T) * E, 0.0);
  oracle_router_dlogits_f64(logits, idx, gate, dgate, T, E, k, renorm, dl.data());
  for (int j = 0; j < d; ++j)
    for (int e = 0; e < E; ++e) {
      double s = 0.0;
      for (int64_t t = 0; t < T; ++t) s += x[t * d + j] * dl[t * E + e];
      dw_r[(int64_t)j * E + e] = s;
    }
  for (int64_t t = 0; t < T; ++t)
    for (int j = 0; j < d; ++j) {
      double s = 0.0;
      for (int e = 0; e < E; ++e) s += dl[t * E + e] * w_r[(int64_t)j * E + e];
      dx[t * d + j] = s;
    }
  if (dbias)
    for (int e = 0; e < E; ++e) {
      double s = 0.0;
      for (int64_t t = 0; t < T; ++t) s += dl[t * E + e];
      dbias[e] = s;
    }
}

}  // extern "C"
