// Memory model and memory-aware chunk tuning from the model configuration
// (paper Section 3, Eq. (1) and Eq. (2); Section 4.2, Eq. (8), Eq. (9) and
// the bin thresholds).  Host arithmetic only, exact in 128-bit integers.
#include <stdint.h>

#include <algorithm>

#include "memfine.h"

namespace {

typedef __int128 i128;
constexpr i128 kI64Max = (i128)INT64_MAX;

bool model_ok(const memfine_model* m) {
  if (!m) return false;
  if (m->b < 1 || m->s < 0 || m->h < 0 || m->a < 0 || m->h_d < 0 || m->k_a < 0 || m->e_n < 0 ||
      m->g_e < 0)
    return false;
  if (m->t < 1 || m->c < 1 || m->v < 1 || m->p < 1 || m->D_t < 1) return false;
  return m->full_recompute == 0 || m->full_recompute == 1;
}

// m_g of Section 3 at pipeline rank r: 1 under full recomputation, else
// v p + p - 2 r - 1; 0 signals an invalid rank.
int64_t m_g(const memfine_model* m, int32_t r) {
  if (r < 0 || r >= m->p) return 0;
  if (m->full_recompute) return 1;
  const int64_t v = (int64_t)m->v * m->p + m->p - 2 * (int64_t)r - 1;
  return v >= 1 ? v : 0;
}

// The per-token part of Eq. (2) that does not depend on s' (elements per
// token and micro-batch row) and the per-slot part.
i128 fixed_width(const memfine_model* m) {
  return 5 * (i128)m->h + (i128)m->a * m->h_d + 2 * (i128)m->k_a * m->h_d + m->e_n;
}
i128 slot_width(const memfine_model* m) { return 2 * (i128)m->h + 2 * (i128)m->g_e; }

i128 ceil_div(i128 a, i128 b) { return a >= 0 ? (a + b - 1) / b : -((-a) / b); }

}  // namespace

extern "C" {

int memfine_static_memory(const int64_t* S_para, int32_t m_n, int32_t v, int32_t l,
                          int32_t D_para, int32_t D_grad, int32_t D_opt, int64_t* bytes_out) {
  if (!bytes_out || m_n < 0 || (m_n > 0 && !S_para) || v < 1 || l < 1 || D_para < 0 ||
      D_grad < 0 || D_opt < 0)
    return MEMFINE_ERR_INVALID_ARG;
  i128 sum = 0;
  for (int32_t i = 0; i < m_n; ++i) {
    if (S_para[i] < 0) return MEMFINE_ERR_INVALID_ARG;
    sum += S_para[i];
  }
  // parameters + gradients + 4 optimizer-state copies, for v stages of l layers
  const i128 per = (i128)D_para + D_grad + 4 * (i128)D_opt;
  const i128 total = per * v * l * sum;
  if (total > kI64Max) return MEMFINE_ERR_INVALID_ARG;
  *bytes_out = (int64_t)total;
  return MEMFINE_OK;
}

int memfine_activation_memory(const memfine_model* m, int32_t r_pp, int64_t s_recv,
                              int64_t* bytes_out) {
  if (!model_ok(m) || !bytes_out || s_recv < 0) return MEMFINE_ERR_INVALID_ARG;
  const int64_t mg = m_g(m, r_pp);
  if (mg < 1) return MEMFINE_ERR_INVALID_ARG;
  // m_g / (t c) * D_t b (s * fixed + s' * slot)
  const i128 num = (i128)mg * m->D_t * m->b * ((i128)m->s * fixed_width(m) + (i128)s_recv * slot_width(m));
  const i128 v = ceil_div(num, (i128)m->t * m->c);
  if (v > kI64Max) return MEMFINE_ERR_INVALID_ARG;
  *bytes_out = (int64_t)v;
  return MEMFINE_OK;
}

int memfine_mact_thresholds(const memfine_model* m, int32_t r_pp, int64_t M_gpu, int64_t alpha_num,
                            int64_t alpha_den, int64_t M_sta, const int32_t* bins, int32_t nbins,
                            int64_t* thresholds_out) {
  if (!model_ok(m) || !bins || nbins < 1 || !thresholds_out || M_gpu < 0 || M_sta < 0 ||
      alpha_num < 0 || alpha_den < 1)
    return MEMFINE_ERR_INVALID_ARG;
  for (int32_t i = 0; i < nbins; ++i)
    if (bins[i] < 1) return MEMFINE_ERR_INVALID_ARG;
  const int64_t mg = m_g(m, r_pp);
  if (mg < 1) return MEMFINE_ERR_INVALID_ARG;
  // Eq. (8) over the common denominator t c alpha_den:
  //   s'_max = N / D,  N = t c (alpha_num M_gpu - alpha_den M_sta)
  //                        - alpha_den m_g D_t b s fixed
  //                    D = alpha_den m_g D_t b slot
  const i128 tc = (i128)m->t * m->c;
  const i128 scale = (i128)alpha_den * mg * m->D_t * m->b;
  const i128 N = tc * ((i128)alpha_num * M_gpu - (i128)alpha_den * M_sta) - scale * m->s * fixed_width(m);
  const i128 D = scale * slot_width(m);
  for (int32_t i = 0; i < nbins; ++i) {
    i128 th;
    if (N < 0) th = -1;                       // Eq. (3) fails before any slot
    else if (D == 0) th = kI64Max;            // slots cost nothing
    else th = (i128)bins[i] * N / D;          // s'' <= bins[i] * s'_max
    thresholds_out[i] = (int64_t)std::min(th, kI64Max);
  }
  return MEMFINE_OK;
}

int memfine_mact_select(const int32_t* bins, const int64_t* thresholds, int32_t nbins,
                        int64_t s_recv, int32_t* chunks_out) {
  if (!bins || !thresholds || nbins < 1 || !chunks_out || s_recv < 0) return MEMFINE_ERR_INVALID_ARG;
  int32_t best = INT32_MAX, largest = 0;
  for (int32_t i = 0; i < nbins; ++i) {
    if (bins[i] < 1) return MEMFINE_ERR_INVALID_ARG;
    largest = std::max(largest, bins[i]);
    if (s_recv <= thresholds[i]) best = std::min(best, bins[i]);
  }
  if (best == INT32_MAX) {
    *chunks_out = largest;
    return MEMFINE_ERR_BUDGET;
  }
  *chunks_out = best;
  return MEMFINE_OK;
}

}  // extern "C"
