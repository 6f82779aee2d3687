/*
 * Speedup and cost model of layer-wise replication (host arithmetic).
 *
 * Sec. 4.2 models a replica set by the number N of consecutive layers it
 * replicates and its parallelism P (1 host + P-1 replica devices):
 *   C_mem(N, P)  = N * kappa * (12 d^2 + bs/P * l * d)      per device
 *   C_comp(N, P) = N/P * 24 * bs * l * d^2                  per device
 *   T(P)         = 2 * (bs/P * (P-1) * l * d * kappa) / B   boundary scatter + gather
 *   W(N, P)      = (L-N) t + N t / P
 *   S(N, P)      = L t / (W(N, P) + T(P))
 * and, per layer with a parallelism vector v[L] over devices of speed t_k:
 *   W(v) = sum_l max_{k < v_l} t_k * ceil(bs / v_l) / bs
 *   T(v) = sum over l with v_l != v_{l+1} (v_L = 1) of 2 ceil(bs (v_l-1)/v_l) l d kappa / B_min
 *   S(v) = L t_0 / (W(v) + T(v))
 * Sec. 4.4 ranks candidate spans for a scaling step by the L1 distance of
 * their vectors to the current one. Where the paper is silent this follows
 * fixed readings: bytes per element and l are explicit in T; layer l runs on
 * devices 0 .. v_l-1 (device 0 the host); a step's device cost is P-1; ties
 * in the ranking go to the larger speedup, then the smaller P, then the
 * smaller N.
 *
 * All functions are pure host code: no GPU, no allocation, thread-safe.
 */
#ifndef COCO_SCALING_H
#define COCO_SCALING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Model inputs shared by the functions below. */
typedef struct {
  int32_t n_layers;        /* L, layers of the model */
  int64_t batch;           /* bs, rows (requests) of the step */
  int64_t tokens_per_row;  /* l: 1 in decode, the chunk length in prefill */
  int64_t d_hidden;        /* d */
  double elem_bytes;       /* kappa: bytes per element (2 for bf16) */
  double t_comp;           /* seconds per layer for the whole batch on one device */
  double bandwidth;        /* B, bytes per second of the boundary link */
} coco_scale_model;

/* Rows per device when bs rows are split over v devices (Sec. 3.1's 15 ->
 * 8 + 7; Sec. 4.2: the heaviest device gets ceil(bs/v), the others floor):
 * the first bs mod v devices get ceil(bs/v). sizes[v] is written.
 * COCO_EINVAL (-1) for bs < 0, v < 1 or a NULL pointer. */
int coco_split_batch(int64_t bs, int32_t v, int64_t* sizes);

/* T(P) in seconds; 0 for P = 1. NaN for a NULL model or P < 1. */
double coco_comm_time(const coco_scale_model* m, int32_t P);

/* S(N, P) = L t / (W(N, P) + T(P)) for 0 <= N <= L, P >= 1 (T = 0 when
 * N = 0 or P = 1). NaN when the arguments are out of range. */
double coco_speedup(const coco_scale_model* m, int32_t N, int32_t P);

/* C_mem(N, P) in bytes and C_comp(N, P) in flops, per device. */
double coco_cost_mem(const coco_scale_model* m, int32_t N, int32_t P);
double coco_cost_comp(const coco_scale_model* m, int32_t N, int32_t P);

/* S(v) for a host vector v[L] (1 <= v_l <= n_dev), device times t_dev[n_dev]
 * (t_dev[0] the host) and link bandwidths bw[n_dev] (B_min = their minimum).
 * NaN on invalid input. */
double coco_speedup_vec(const coco_scale_model* m, const int32_t* v, const double* t_dev,
                        const double* bw, int32_t n_dev);

/* One candidate of a scaling step. */
typedef struct {
  int32_t n_layers;   /* N (0 for no replication) */
  int32_t parallel;   /* P */
  double speedup;     /* S(N, P) */
  int32_t distance;   /* L1 distance of its vector to the current one */
} coco_scale_candidate;

/* The unified scaling step of Sec. 4.4 for one instance whose replicated
 * span starts at layer `first`: alpha_req = S(n_cur, p_cur) *
 * latency_over_slo; the candidates (0, 1) and (N, P) with 1 <= N <= L-first,
 * 2 <= P <= p_max, whose S reaches alpha_req, ranked as above, are written to
 * out[max_out] (*n_out = how many qualify, possibly more than max_out);
 * *chosen = index in the ranking of the first candidate whose extra replica
 * devices (P-1) - (p_cur-1) are <= 0 or fit in cold_devices, -1 if none.
 * COCO_EINVAL for invalid arguments. */
int coco_scale_candidates(const coco_scale_model* m, int32_t first, int32_t p_max,
                          int32_t n_cur, int32_t p_cur, double latency_over_slo,
                          int32_t cold_devices, coco_scale_candidate* out, int32_t max_out,
                          int32_t* n_out, int32_t* chosen, double* alpha_req);

#ifdef __cplusplus
}
#endif

#endif /* COCO_SCALING_H */
