// Host planner: the static, weight-derived selection plan of DASC.
//
//   Sec. 3.3, Eq. 2  g = -exp(A_log) * softplus(a + dt_bias), a = -0.3
//   Sec. 3.3, Eq. 3  H_s = ln(eps) / g
//   Sec. 4.1         retain unit u iff H_s(u) > W_max (KDA unit = key-channel row,
//                    GDN unit = head); Eq. 6 compression ratios, padded layout
//   App. B           ragged offsets o_0 = 0, o_{l+1} = o_l + r_l
//   Sec. 4.2, Eq. 7  W_u = clamp(next_pow2(H_s(u)), 4, W_max), W_replay = max over omitted
//   Sec. 4.3         balanced per-rank slot width C = ceil(sum_r U_r / T)
//   App. C.1, Eq. 8  matched-HBM slot count N = floor(B / b) - 1
//
// Built without fast-math or FP contraction: every value is produced by the same
// sequence of IEEE binary64 operations and libm calls as a straightforward reading
// of those equations, so identical inputs give identical bits on every call.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <numeric>
#include <vector>

#include "dasc.h"

namespace {

double softplus(double x) { return std::max(x, 0.0) + std::log1p(std::exp(-std::fabs(x))); }

int64_t next_pow2(double x) {
  int64_t p = 1;
  while (static_cast<double>(p) < x) p *= 2;
  return p;
}

int32_t replay_window(double h, int32_t w_max) {
  if (h >= static_cast<double>(w_max)) return w_max;  // next_pow2(h) >= h >= W_max
  int64_t p = std::max<int64_t>(next_pow2(h), 4);
  return static_cast<int32_t>(std::min<int64_t>(p, w_max));
}

bool shape_ok(const dasc_shape& s) {
  if (s.arch != DASC_ARCH_KDA && s.arch != DASC_ARCH_GDN) return false;
  if (s.n_layers <= 0 || s.n_heads <= 0 || s.n_qk_heads <= 0 || s.dk <= 0 || s.dv <= 0) return false;
  if (s.n_heads % s.n_qk_heads != 0) return false;
  const int64_t rows = int64_t(s.n_layers) * s.n_heads * s.dk;
  return rows < (int64_t(1) << 31);
}

}  // namespace

extern "C" int dasc_static_log_decay(const double* a_log, const double* dt_bias, double a,
                                     int64_t n, double* g_out) {
  if (!a_log || !g_out || n < 0) return DASC_E_INVAL;
  for (int64_t i = 0; i < n; ++i) {
    const double dt = dt_bias ? dt_bias[i] : 0.0;
    g_out[i] = -std::exp(a_log[i]) * softplus(a + dt);
  }
  return DASC_OK;
}

extern "C" int dasc_matched_slots(int64_t budget_bytes, int64_t slot_bytes, int64_t* slots) {
  if (!slots || budget_bytes < 0 || slot_bytes <= 0) return DASC_E_INVAL;
  *slots = budget_bytes / slot_bytes - 1;
  return DASC_OK;
}

extern "C" int dasc_plan(const dasc_plan_desc* desc, const double* g, dasc_plan_out* out) {
  if (!desc || !g || !out) return DASC_E_INVAL;
  const dasc_shape& s = desc->shape;
  if (!shape_ok(s)) return DASC_E_SHAPE;
  const bool kda = s.arch == DASC_ARCH_KDA;
  const int64_t L = s.n_layers, H = s.n_heads, dk = s.dk, dv = s.dv;
  const int64_t n_lh = L * H;
  const int64_t n_rows_dense = n_lh * dk;
  const int64_t n_per_layer = kda ? H * dk : H;
  const int64_t n_units_total = L * n_per_layer;
  if (!(desc->eps > 0.0 && desc->eps < 1.0)) return DASC_E_INVAL;
  if (desc->w_max < 0 || desc->n_ranks < 1 || desc->conv_bytes < 0) return DASC_E_INVAL;
  switch (desc->keep_mode) {
    case DASC_KEEP_THRESHOLD: break;
    case DASC_KEEP_TOPK_PER_HEAD:
      if (!kda) return DASC_E_SHAPE;
      if (desc->keep_k < 0 || desc->keep_k > dk) return DASC_E_INVAL;
      break;
    case DASC_KEEP_TOPK_PER_LAYER:
      if (desc->keep_k < 0 || desc->keep_k > n_per_layer) return DASC_E_INVAL;
      break;
    default: return DASC_E_INVAL;
  }
  for (int64_t u = 0; u < n_units_total; ++u)
    if (!std::isfinite(g[u]) || !(g[u] < 0.0)) return DASC_E_INVAL;

  // Eq. 3
  const double ln_eps = std::log(desc->eps);
  std::vector<double> hs(n_units_total);
  for (int64_t u = 0; u < n_units_total; ++u) hs[u] = ln_eps / g[u];

  // Sec. 4.1 selection
  std::vector<uint8_t> keep(n_units_total, 0);
  auto keep_top = [&](int64_t first, int64_t count, int64_t k) {
    std::vector<int64_t> idx(count);
    std::iota(idx.begin(), idx.end(), int64_t(0));
    std::sort(idx.begin(), idx.end(), [&](int64_t a, int64_t b) {
      const double ha = hs[first + a], hb = hs[first + b];
      return ha > hb || (ha == hb && a < b);
    });
    for (int64_t i = 0; i < k; ++i) keep[first + idx[i]] = 1;
  };
  if (desc->keep_mode == DASC_KEEP_THRESHOLD) {
    const double w = static_cast<double>(desc->w_max);
    for (int64_t u = 0; u < n_units_total; ++u) keep[u] = hs[u] > w ? 1 : 0;
  } else if (desc->keep_mode == DASC_KEEP_TOPK_PER_HEAD) {
    for (int64_t lh = 0; lh < n_lh; ++lh) keep_top(lh * dk, dk, desc->keep_k);
  } else {
    for (int64_t l = 0; l < L; ++l) keep_top(l * n_per_layer, n_per_layer, desc->keep_k);
  }

  // kept units per (l, h) and the packed-row maps in (layer, head, channel) order
  const int64_t rows_per_unit = kda ? 1 : dk;
  std::vector<int64_t> ucount(n_lh, 0);
  for (int64_t lh = 0; lh < n_lh; ++lh) {
    if (kda) {
      for (int64_t c = 0; c < dk; ++c) ucount[lh] += keep[lh * dk + c];
    } else {
      ucount[lh] = keep[lh];
    }
  }
  int64_t n_rows = 0, n_units = 0;
  for (int64_t lh = 0; lh < n_lh; ++lh) {
    if (out->off) out->off[lh] = static_cast<int32_t>(n_rows);
    if (out->unit_count) out->unit_count[lh] = static_cast<int32_t>(ucount[lh]);
    n_rows += ucount[lh] * rows_per_unit;
    n_units += ucount[lh];
  }
  if (out->off) out->off[n_lh] = static_cast<int32_t>(n_rows);

  if (out->unit_row || out->inv_row) {
    int64_t j = 0;
    for (int64_t lh = 0; lh < n_lh; ++lh) {
      for (int64_t c = 0; c < dk; ++c) {
        const int64_t dense = lh * dk + c;
        const bool kept = kda ? keep[dense] : keep[lh];
        if (out->inv_row) out->inv_row[dense] = kept ? static_cast<int32_t>(j) : -1;
        if (kept) {
          if (out->unit_row) out->unit_row[j] = static_cast<int32_t>(dense);
          ++j;
        }
      }
    }
  }

  // App. B per-layer offsets (units)
  std::vector<int64_t> r_layer(L, 0);
  for (int64_t l = 0; l < L; ++l)
    for (int64_t h = 0; h < H; ++h) r_layer[l] += ucount[l * H + h];
  if (out->layer_off || out->layer_off_rows) {
    int64_t acc = 0;
    if (out->layer_off) out->layer_off[0] = 0;
    if (out->layer_off_rows) out->layer_off_rows[0] = 0;
    for (int64_t l = 0; l < L; ++l) {
      acc += r_layer[l];
      if (out->layer_off) out->layer_off[l + 1] = static_cast<int32_t>(acc);
      if (out->layer_off_rows) out->layer_off_rows[l + 1] = static_cast<int32_t>(acc * rows_per_unit);
    }
  }

  // Eq. 7
  int32_t w_replay = 0;
  for (int64_t u = 0; u < n_units_total; ++u) {
    int32_t w = 0;
    if (!keep[u]) {
      w = replay_window(hs[u], desc->w_max);
      w_replay = std::max(w_replay, w);
    }
    if (out->w_units) out->w_units[u] = w;
  }

  // Sec. 4.3 slices and send matrix
  const int64_t T = desc->n_ranks;
  const int64_t C = (n_units + T - 1) / T;
  if (out->rank_begin)
    for (int64_t r = 0; r <= T; ++r)
      out->rank_begin[r] = static_cast<int32_t>(std::min(r * C, n_units) * rows_per_unit);
  if (out->send) {
    std::memset(out->send, 0, sizeof(int64_t) * T * T);
    int64_t p = 0;
    for (int64_t l = 0; l < L; ++l)
      for (int64_t h = 0; h < H; ++h) {
        const int64_t owner = (h * T) / H;
        for (int64_t i = 0; i < ucount[l * H + h]; ++i, ++p) out->send[owner * T + p / C] += 1;
      }
  }

  // Eq. 6 and the padded layout
  const double inf = std::numeric_limits<double>::infinity();
  const int64_t sum_n = L * n_per_layer;
  const int64_t r_max = *std::max_element(r_layer.begin(), r_layer.end());
  const double r_bar = static_cast<double>(n_units) / static_cast<double>(L);
  const int64_t unit_bytes = rows_per_unit * dv * 4;
  const int64_t dense_rank = ((sum_n + T - 1) / T) * unit_bytes;
  const int64_t rag_rank = C * unit_bytes;
  out->c_temp_rag = n_units ? static_cast<double>(sum_n) / static_cast<double>(n_units) : inf;
  out->c_temp_pad = r_max ? static_cast<double>(sum_n) / static_cast<double>(L * r_max) : inf;
  out->layout_gain = n_units ? static_cast<double>(r_max) / r_bar : std::numeric_limits<double>::quiet_NaN();
  out->c_ckpt = (rag_rank + desc->conv_bytes)
                    ? static_cast<double>(dense_rank + desc->conv_bytes) /
                          static_cast<double>(rag_rank + desc->conv_bytes)
                    : inf;
  out->r_max_rows = r_max * rows_per_unit;
  out->slot_bytes_rank = rag_rank + desc->conv_bytes;
  out->dense_slot_bytes_rank = dense_rank + desc->conv_bytes;

  if (out->keep) std::memcpy(out->keep, keep.data(), n_units_total);
  if (out->horizon) std::memcpy(out->horizon, hs.data(), sizeof(double) * n_units_total);
  out->n_rows = n_rows;
  out->n_units = n_units;
  out->rows_per_unit = static_cast<int32_t>(rows_per_unit);
  out->w_replay = w_replay;
  out->slice_units = C;
  out->slice_rows = C * rows_per_unit;
  (void)n_rows_dense;
  return DASC_OK;
}

extern "C" int dasc_tp_permutation(const dasc_shape* shape, const int32_t* unit_count,
                                   int32_t n_ranks, int32_t* head_perm, int64_t* rank_rows,
                                   int64_t* rank_rows_identity) {
  if (!shape) return DASC_E_SHAPE;
  if (shape->arch != DASC_ARCH_KDA && shape->arch != DASC_ARCH_GDN) return DASC_E_SHAPE;
  const int L = shape->n_layers, H = shape->n_heads, B = shape->n_qk_heads;
  if (L <= 0 || H <= 0 || B <= 0 || shape->dk <= 0 || shape->dv <= 0 || H % B != 0)
    return DASC_E_SHAPE;
  if (int64_t(L) * H * shape->dk >= (int64_t(1) << 31)) return DASC_E_SHAPE;
  if (!unit_count || !head_perm || !rank_rows || !rank_rows_identity) return DASC_E_INVAL;
  if (n_ranks < 1 || B % n_ranks != 0) return DASC_E_INVAL;
  const bool kda = shape->arch == DASC_ARCH_KDA;
  const int max_units = kda ? shape->dk : 1;
  for (int64_t i = 0; i < int64_t(L) * H; ++i)
    if (unit_count[i] < 0 || unit_count[i] > max_units) return DASC_E_INVAL;

  const int T = n_ranks, g = H / B, cap = B / T;
  const int64_t rows_per_unit = kda ? 1 : shape->dk;
  std::vector<int64_t> load(size_t(L) * B, 0);    // retained rows per (layer, bundle)
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < B; ++b) {
      int64_t units = 0;
      for (int i = 0; i < g; ++i) units += unit_count[int64_t(l) * H + b * g + i];
      load[size_t(l) * B + b] = units * rows_per_unit;
    }
  std::vector<int64_t> ident(T, 0);
  for (int l = 0; l < L; ++l)
    for (int b = 0; b < B; ++b) ident[b / cap] += load[size_t(l) * B + b];

  std::vector<int> order(size_t(L) * B);
  for (size_t i = 0; i < order.size(); ++i) order[i] = int(i);
  // largest first; ties to the lower (layer, bundle), which is the lower flat index
  std::stable_sort(order.begin(), order.end(),
                   [&](int a, int b) { return load[a] > load[b]; });
  std::vector<int64_t> U(T, 0);
  std::vector<int> used(size_t(L) * T, 0), owner(size_t(L) * B, 0);
  for (int item : order) {
    const int l = item / B;
    int best = -1;
    for (int r = 0; r < T; ++r)
      if (used[size_t(l) * T + r] < cap && (best < 0 || U[r] < U[best])) best = r;
    owner[item] = best;
    ++used[size_t(l) * T + best];
    U[best] += load[item];
  }
  if (*std::max_element(U.begin(), U.end()) >= *std::max_element(ident.begin(), ident.end())) {
    for (int l = 0; l < L; ++l)
      for (int b = 0; b < B; ++b) owner[size_t(l) * B + b] = b / cap;
    U = ident;
  }
  for (int l = 0; l < L; ++l) {
    int pos = 0;
    for (int r = 0; r < T; ++r)
      for (int b = 0; b < B; ++b)
        if (owner[size_t(l) * B + b] == r)
          for (int i = 0; i < g; ++i) head_perm[int64_t(l) * H + pos++] = b * g + i;
  }
  for (int r = 0; r < T; ++r) {
    rank_rows[r] = U[r];
    rank_rows_identity[r] = ident[r];
  }
  return DASC_OK;
}

extern "C" const char* dasc_strerror(int code) {
  switch (code) {
    case DASC_OK: return "ok";
    case DASC_E_INVAL: return "invalid argument (null pointer, misalignment or value out of range)";
    case DASC_E_SHAPE: return "inconsistent shape";
    case DASC_E_WORKSPACE: return "workspace too small";
    case DASC_E_HIP: return "HIP runtime error at launch";
    case DASC_E_UNSUPPORTED: return "no kernel built for this shape";
    case DASC_E_SCRATCH:
      return "request needs more scratch than dasc_refresh_noalloc holds "
             "(DASC_NOALLOC_SCRATCH_BYTES); use dasc_refresh with a workspace";
    default: return "unknown status code";
  }
}
