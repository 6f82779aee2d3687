// Speedup and cost model of layer-wise replication (Sec. 4.2) and the
// candidate ranking of the unified scaling step (Sec. 4.4). Host arithmetic
// only; the formulas and readings are listed in coco_scaling.h.
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <vector>

#include "../../include/coco.h"
#include "../../include/coco_scaling.h"

namespace {

bool model_ok(const coco_scale_model* m) {
  return m && m->n_layers >= 1 && m->batch >= 1 && m->tokens_per_row >= 1 &&
         m->d_hidden >= 1 && m->elem_bytes > 0 && m->t_comp > 0 && m->bandwidth > 0;
}

// T(P): the (P-1)/P share of the rows leaves at the span's start and comes
// back at its end.
double comm(const coco_scale_model& m, int32_t P) {
  const double moved = (double)m.batch / P * (P - 1) * (double)m.tokens_per_row *
                       (double)m.d_hidden * m.elem_bytes;
  return 2.0 * moved / m.bandwidth;
}

double span_speedup(const coco_scale_model& m, int32_t N, int32_t P) {
  const int32_t L = m.n_layers;
  const double t = m.t_comp;
  const double w = (double)(L - N) * t + (double)N * t / P;
  const double T = N > 0 ? comm(m, P) : 0.0;
  return (double)L * t / (w + T);
}

// Parallelism of layer i for a span of N layers at P starting at `first`.
inline int32_t span_at(int32_t i, int32_t first, int32_t N, int32_t P) {
  return (i >= first && i < first + N) ? P : 1;
}

}  // namespace

extern "C" {

int coco_split_batch(int64_t bs, int32_t v, int64_t* sizes) {
  if (bs < 0 || v < 1 || !sizes) return COCO_EINVAL;
  const int64_t base = bs / v, extra = bs % v;
  for (int32_t k = 0; k < v; ++k) sizes[k] = base + (k < extra ? 1 : 0);
  return COCO_OK;
}

double coco_comm_time(const coco_scale_model* m, int32_t P) {
  if (!model_ok(m) || P < 1) return NAN;
  return comm(*m, P);
}

double coco_speedup(const coco_scale_model* m, int32_t N, int32_t P) {
  if (!model_ok(m) || P < 1 || N < 0 || N > m->n_layers) return NAN;
  return span_speedup(*m, N, P);
}

double coco_cost_mem(const coco_scale_model* m, int32_t N, int32_t P) {
  if (!model_ok(m) || P < 1 || N < 0) return NAN;
  const double d = (double)m->d_hidden;
  return (double)N * m->elem_bytes *
         (12.0 * d * d + (double)m->batch / P * (double)m->tokens_per_row * d);
}

double coco_cost_comp(const coco_scale_model* m, int32_t N, int32_t P) {
  if (!model_ok(m) || P < 1 || N < 0) return NAN;
  const double d = (double)m->d_hidden;
  return (double)N / P * 24.0 * (double)m->batch * (double)m->tokens_per_row * d * d;
}

double coco_speedup_vec(const coco_scale_model* m, const int32_t* v, const double* t_dev,
                        const double* bw, int32_t n_dev) {
  if (!model_ok(m) || !v || !t_dev || !bw || n_dev < 1) return NAN;
  const int32_t L = m->n_layers;
  const int64_t bs = m->batch;
  double b_min = bw[0];
  for (int32_t k = 1; k < n_dev; ++k) b_min = std::min(b_min, bw[k]);
  if (!(b_min > 0)) return NAN;
  double w = 0.0, T = 0.0;
  for (int32_t i = 0; i < L; ++i) {
    const int32_t vl = v[i];
    if (vl < 1 || vl > n_dev) return NAN;
    double slowest = t_dev[0];
    for (int32_t k = 1; k < vl; ++k) slowest = std::max(slowest, t_dev[k]);
    const int64_t heaviest = (bs + vl - 1) / vl;  // ceil(bs / v_l)
    w += slowest * (double)heaviest / (double)bs;
    const int32_t next = i + 1 < L ? v[i + 1] : 1;
    if (vl != next) {
      const int64_t rows = (bs * (vl - 1) + vl - 1) / vl;  // ceil(bs (v_l - 1) / v_l)
      T += 2.0 * (double)rows * (double)m->tokens_per_row * (double)m->d_hidden *
           m->elem_bytes / b_min;
    }
  }
  return (double)L * t_dev[0] / (w + T);
}

int coco_scale_candidates(const coco_scale_model* m, int32_t first, int32_t p_max,
                          int32_t n_cur, int32_t p_cur, double latency_over_slo,
                          int32_t cold_devices, coco_scale_candidate* out, int32_t max_out,
                          int32_t* n_out, int32_t* chosen, double* alpha_req) {
  if (!model_ok(m) || first < 0 || first >= m->n_layers || p_max < 1 || p_cur < 1 ||
      p_cur > p_max || n_cur < 0 || first + n_cur > m->n_layers ||
      !(latency_over_slo > 0) || cold_devices < 0 || max_out < 0 ||
      (max_out > 0 && !out) || !n_out || !chosen || !alpha_req)
    return COCO_EINVAL;
  const int32_t L = m->n_layers;
  const double alpha = span_speedup(*m, n_cur, p_cur) * latency_over_slo;

  std::vector<coco_scale_candidate> c;
  auto consider = [&](int32_t N, int32_t P) {
    const double s = span_speedup(*m, N, P);
    if (!(s >= alpha)) return;
    int32_t dist = 0;
    for (int32_t i = 0; i < L; ++i) {
      const int32_t a = span_at(i, first, n_cur, p_cur), b = span_at(i, first, N, P);
      dist += a > b ? a - b : b - a;
    }
    c.push_back(coco_scale_candidate{N, P, s, dist});
  };
  consider(0, 1);
  for (int32_t P = 2; P <= p_max; ++P)
    for (int32_t N = 1; N <= L - first; ++N) consider(N, P);
  std::stable_sort(c.begin(), c.end(),
                   [](const coco_scale_candidate& x, const coco_scale_candidate& y) {
                     if (x.distance != y.distance) return x.distance < y.distance;
                     if (x.speedup != y.speedup) return x.speedup > y.speedup;
                     if (x.parallel != y.parallel) return x.parallel < y.parallel;
                     return x.n_layers < y.n_layers;
                   });
  int32_t pick = -1;
  for (size_t i = 0; i < c.size(); ++i) {
    const int32_t extra = (c[i].parallel - 1) - (p_cur - 1);
    if (extra <= 0 || cold_devices >= extra) {
      pick = (int32_t)i;
      break;
    }
  }
  for (int32_t i = 0; i < max_out && i < (int32_t)c.size(); ++i) out[i] = c[i];
  *n_out = (int32_t)c.size();
  *chosen = pick;
  *alpha_req = alpha;
  return COCO_OK;
}

}  // extern "C"
