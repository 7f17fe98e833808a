/*
 * fgref.c -- plain CPU oracle for FeatGraph's generalized SpMM, generalized
 * SDDMM and the edge softmax that links them in an attention layer.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code,
 * header or constant with the GPU library; it is deliberately slow and
 * written so that each function can be checked against the paper by eye.
 *
 * Graph convention: CSR whose rows are destination vertices.  For row v the
 * stored edges are p = indptr[v] .. indptr[v+1]-1 in storage order, the
 * source vertex is u = indices[p] and the edge id is e = edge_ids[p] (or p
 * when edge_ids is NULL).  Vertex data is row-major [vertices, H, dh]; edge
 * data is row-major [edge id, H].
 *
 * Precision: inputs and outputs are fp32; sums and dot products accumulate
 * in fp64 and are rounded to fp32 once.  Where a float comparison decides an
 * index (max / argmax) the compared message is the fp32 value, exactly as
 * the GPU path sees it.
 *
 * Threading: rows are independent, each row is computed by one thread in a
 * fixed order, so results do not depend on the thread count.
 *
 * Return value of every entry point: 0 on success, a negative number for
 * invalid arguments (nothing written in that case).
 */
#include <math.h>
#include <stddef.h>
#include <stdlib.h>
#include <stdint.h>
#include <omp.h>

#define FGREF_EXPORT __attribute__((visibility("default")))

enum { MSG_COPY_SRC = 0, MSG_SRC_MUL_EDGE = 1 };
enum { RED_SUM = 0, RED_MAX = 1 };

static int set_threads(int num_threads) {
  if (num_threads > 0) omp_set_num_threads(num_threads);
  return 0;
}

/* Row of the i-th selected output: either rows[i] or i itself. */
static int64_t pick_row(const int64_t* rows, int64_t i) { return rows ? rows[i] : i; }

static int check_rows(const int64_t* rows, int64_t num_sel, int64_t num_rows) {
  if (!rows) return 0;
  for (int64_t i = 0; i < num_sel; ++i)
    if (rows[i] < 0 || rows[i] >= num_rows) return -1;
  return 0;
}

/*
 * Generalized SpMM (Sec. II-A Eq. 1: h_v = (+)_{u in N(v)} phi(x_u, x_v, x_uv);
 * Eq. 3 is the case phi = copy source, (+) = sum).  The message function phi
 * is one of
 *   copy_src      : m = X[u, h, k]
 *   src_mul_edge  : m = (float)(W[e, h] * X[u, h, k])   (product rounded to fp32)
 * and the aggregator (+) is sum or max (Sec. III-B: any commutative reducer).
 *
 * sum : out[v,h,k] = (float) sum_p (double) m            (empty row -> 0)
 * max : out[v,h,k] = max_p m, arg[v,h,k] = the smallest edge id attaining it;
 *       empty row -> out 0, arg -1.  Equality is IEEE equality, so -0 == +0
 *       and the edge id decides between them.  A NaN message takes part as
 *       -inf (the paper leaves NaN undefined; this is the library's reading),
 *       so it never beats a number and a row of NaN / -inf messages gives
 *       -inf with its smallest edge id.
 *
 * Output i (0 <= i < num_sel) is row pick_row(rows, i); with rows == NULL all
 * num_rows rows are computed (num_sel must then equal num_rows).
 * term_norm (optional, sum only) receives sqrt(sum_p m^2) per output element.
 */
FGREF_EXPORT int fgref_gspmm(int64_t num_rows, int64_t num_cols, const int32_t* indptr,
                             const int32_t* indices, const int32_t* edge_ids, int64_t nnz_total,
                             int msg, int red, int64_t H, int64_t dh, const float* x,
                             const float* edge_val, const int64_t* rows, int64_t num_sel,
                             float* out, int32_t* arg, double* term_norm, int num_threads) {
  if (H < 1 || dh < 1 || num_rows < 0 || num_cols < 0 || !indptr || !out) return -1;
  if (msg != MSG_COPY_SRC && msg != MSG_SRC_MUL_EDGE) return -1;
  if (red != RED_SUM && red != RED_MAX) return -1;
  if (msg == MSG_SRC_MUL_EDGE && !edge_val) return -1;
  if (red == RED_MAX && !arg) return -1;
  if (!rows && num_sel != num_rows) return -1;
  if (check_rows(rows, num_sel, num_rows)) return -1;
  set_threads(num_threads);
  const int64_t F = H * dh;
  int bad = 0;

#pragma omp parallel for schedule(dynamic, 64) reduction(| : bad)
  for (int64_t i = 0; i < num_sel; ++i) {
    const int64_t v = pick_row(rows, i);
    const int64_t p0 = indptr[v], p1 = indptr[v + 1];
    for (int64_t h = 0; h < H; ++h) {
      for (int64_t k = 0; k < dh; ++k) {
        const int64_t f = h * dh + k;
        double acc = 0.0, sq = 0.0;
        float best = 0.0f;
        int32_t best_e = -1;
        for (int64_t p = p0; p < p1; ++p) {
          const int64_t u = indices[p];
          const int64_t e = edge_ids ? edge_ids[p] : p;
          if (u < 0 || u >= num_cols || e < 0 || e >= nnz_total) { bad |= 1; continue; }
          float m = x[u * F + f];
          if (msg == MSG_SRC_MUL_EDGE) m = edge_val[e * H + h] * m;
          if (red == RED_MAX && isnan(m)) m = -INFINITY;
          if (red == RED_SUM) {
            acc += (double)m;
            sq += (double)m * (double)m;
          } else if (best_e == -1 || m > best || (m == best && e < best_e)) {
            best = m;
            best_e = (int32_t)e;
          }
        }
        if (red == RED_SUM) {
          out[i * F + f] = (float)acc;
          if (term_norm) term_norm[i * F + f] = sqrt(sq);
        } else {
          out[i * F + f] = best_e == -1 ? 0.0f : best;
          arg[i * F + f] = best_e;
        }
      }
    }
  }
  return bad ? -2 : 0;
}

/*
 * Generalized SDDMM with the dot-product edge function (Sec. II-A Eq. 2 with
 * psi(x_u, x_v, x_uv) = x_u x_v^T, Eq. 4), per head for multi-head attention
 * (Fig. 4b: H dot products of length dh):
 *   out[e, h] = (float) sum_k (double) Xs[u, h, k] * (double) Xd[v, h, k]
 * for every stored edge (v <- u) with id e of the selected rows.  Outputs of
 * edges outside the selected rows are left untouched.  term_norm (optional,
 * indexed like out) receives sqrt(sum_k (Xs*Xd)^2).
 */
FGREF_EXPORT int fgref_gsddmm(int64_t num_rows, int64_t num_cols, const int32_t* indptr,
                              const int32_t* indices, const int32_t* edge_ids, int64_t nnz_total,
                              int64_t H, int64_t dh, const float* xs, const float* xd,
                              const int64_t* rows, int64_t num_sel, float* out, double* term_norm,
                              int num_threads) {
  if (H < 1 || dh < 1 || num_rows < 0 || num_cols < 0 || !indptr || !out) return -1;
  if (!rows && num_sel != num_rows) return -1;
  if (check_rows(rows, num_sel, num_rows)) return -1;
  set_threads(num_threads);
  const int64_t F = H * dh;
  int bad = 0;

#pragma omp parallel for schedule(dynamic, 64) reduction(| : bad)
  for (int64_t i = 0; i < num_sel; ++i) {
    const int64_t v = pick_row(rows, i);
    for (int64_t p = indptr[v]; p < indptr[v + 1]; ++p) {
      const int64_t u = indices[p];
      const int64_t e = edge_ids ? edge_ids[p] : p;
      if (u < 0 || u >= num_cols || e < 0 || e >= nnz_total) { bad |= 1; continue; }
      for (int64_t h = 0; h < H; ++h) {
        double acc = 0.0, sq = 0.0;
        for (int64_t k = 0; k < dh; ++k) {
          const double t = (double)xs[u * F + h * dh + k] * (double)xd[v * F + h * dh + k];
          acc += t;
          sq += t * t;
        }
        out[e * H + h] = (float)acc;
        if (term_norm) term_norm[e * H + h] = sqrt(sq);
      }
    }
  }
  return bad ? -2 : 0;
}

/*
 * Edge softmax over each destination's in-edges, per head, optionally after
 * a leaky ReLU (the attention normalisation of a graph attention layer):
 *   s'  = s > 0 ? s : slope * s           (fp64)
 *   out[e, h] = exp(s'_e - m) / sum_{p in row} exp(s'_p - m),  m = max_p s'_p
 * Subtracting the row maximum does not change the value.  Rows with no edges
 * write nothing.  Computed in fp64 and rounded to fp32 once.
 */
FGREF_EXPORT int fgref_edge_softmax(int64_t num_rows, const int32_t* indptr,
                                    const int32_t* edge_ids, int64_t nnz_total, int64_t H,
                                    const float* scores, int apply_leaky_relu, float slope,
                                    const int64_t* rows, int64_t num_sel, float* out,
                                    int num_threads) {
  if (H < 1 || num_rows < 0 || !indptr || !scores || !out) return -1;
  if (!rows && num_sel != num_rows) return -1;
  if (check_rows(rows, num_sel, num_rows)) return -1;
  set_threads(num_threads);
  int bad = 0;

#pragma omp parallel for schedule(dynamic, 64) reduction(| : bad)
  for (int64_t i = 0; i < num_sel; ++i) {
    const int64_t v = pick_row(rows, i);
    const int64_t p0 = indptr[v], p1 = indptr[v + 1];
    for (int64_t p = p0; p < p1; ++p) {
      const int64_t e = edge_ids ? edge_ids[p] : p;
      if (e < 0 || e >= nnz_total) bad |= 1;
    }
    if (bad) continue;
    for (int64_t h = 0; h < H; ++h) {
      double m = -INFINITY;
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        double s = scores[e * H + h];
        if (apply_leaky_relu && !(s > 0.0)) s = (double)slope * s;
        if (s > m) m = s;
      }
      double z = 0.0;
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        double s = scores[e * H + h];
        if (apply_leaky_relu && !(s > 0.0)) s = (double)slope * s;
        z += exp(s - m);
      }
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        double s = scores[e * H + h];
        if (apply_leaky_relu && !(s > 0.0)) s = (double)slope * s;
        out[e * H + h] = (float)(exp(s - m) / z);
      }
    }
  }
  return bad ? -2 : 0;
}

/*
 * Gradient of gSpMM with the max aggregator (Eq. 1 with (+) = max).  The
 * output out[v,h,k] equals the message of one edge, the one the forward picks
 * (largest message, smallest edge id among equal ones), so for a loss L with
 * upstream gradient G = dL/dout only that edge receives G[v,h,k]:
 *   copy_src     : dX[u,h,k] += G[v,h,k]
 *   src_mul_edge : dX[u,h,k] += W[e,h] * G[v,h,k],  dW[e,h] += X[u,h,k] * G[v,h,k]
 * where e is the selected edge and u its source.  Empty rows contribute
 * nothing.  The argmax is recomputed here from x with fgref_gspmm (not taken
 * from the caller), then the contributions of the selected rows are added in row order
 * in fp64 and rounded to fp32 once.  grad_src [num_cols, F] and grad_edge
 * [nnz_total, H] (src_mul_edge only) are fully overwritten; either may be
 * NULL.  src_norm / edge_norm (optional, same shapes) receive
 * sqrt(sum of squared contributions).  Edge ids must be distinct.
 */
FGREF_EXPORT int fgref_gspmm_max_backward(int64_t num_rows, int64_t num_cols,
                                          const int32_t* indptr, const int32_t* indices,
                                          const int32_t* edge_ids, int64_t nnz_total, int msg,
                                          int64_t H, int64_t dh, const float* x,
                                          const float* edge_val, const float* grad_out,
                                          const int64_t* rows, int64_t num_sel, float* grad_src,
                                          float* grad_edge, double* src_norm, double* edge_norm,
                                          int num_threads) {
  if (H < 1 || dh < 1 || num_rows < 0 || num_cols < 0 || nnz_total < 0 || !indptr) return -1;
  if (msg != MSG_COPY_SRC && msg != MSG_SRC_MUL_EDGE) return -1;
  if (msg == MSG_COPY_SRC && grad_edge) return -1;
  if (msg == MSG_SRC_MUL_EDGE && !edge_val) return -1;
  if (!x || !grad_out || (!rows && num_sel != num_rows)) return -1;
  if (check_rows(rows, num_sel, num_rows)) return -1;
  const int64_t F = H * dh;
  const int64_t nnz = indptr[num_rows];
  int rc = -3;
  float* fwd = (float*)malloc(sizeof(float) * (size_t)(num_sel * F + 1));
  int32_t* arg = (int32_t*)malloc(sizeof(int32_t) * (size_t)(num_sel * F + 1));
  int64_t* pos = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nnz_total + 1));
  double* gs = (double*)calloc((size_t)(num_cols * F + 1), sizeof(double));
  double* gs2 = (double*)calloc((size_t)(num_cols * F + 1), sizeof(double));
  double* ge = (double*)calloc((size_t)(nnz_total * H + 1), sizeof(double));
  double* ge2 = (double*)calloc((size_t)(nnz_total * H + 1), sizeof(double));
  if (!fwd || !arg || !pos || !gs || !gs2 || !ge || !ge2) goto done;

  /* forward: the edge each output element takes its value from */
  rc = fgref_gspmm(num_rows, num_cols, indptr, indices, edge_ids, nnz_total, msg, RED_MAX, H, dh,
                   x, edge_val, rows, num_sel, fwd, arg, NULL, num_threads);
  if (rc != 0) goto done;

  /* storage position of every edge id */
  for (int64_t e = 0; e < nnz_total; ++e) pos[e] = -1;
  for (int64_t p = 0; p < nnz; ++p) {
    const int64_t e = edge_ids ? edge_ids[p] : p;
    if (e < 0 || e >= nnz_total || pos[e] != -1) { rc = -2; goto done; }
    pos[e] = p;
  }

  for (int64_t i = 0; i < num_sel; ++i) {
    const int64_t v = pick_row(rows, i);
    for (int64_t h = 0; h < H; ++h) {
      for (int64_t k = 0; k < dh; ++k) {
        const int64_t f = h * dh + k;
        const int64_t e = arg[i * F + f];
        if (e < 0) continue;
        const int64_t u = indices[pos[e]];
        const double g = grad_out[v * F + f];
        const double ts = msg == MSG_SRC_MUL_EDGE ? (double)edge_val[e * H + h] * g : g;
        gs[u * F + f] += ts;
        gs2[u * F + f] += ts * ts;
        if (msg == MSG_SRC_MUL_EDGE) {
          const double te = (double)x[u * F + f] * g;
          ge[e * H + h] += te;
          ge2[e * H + h] += te * te;
        }
      }
    }
  }
  if (grad_src)
    for (int64_t j = 0; j < num_cols * F; ++j) grad_src[j] = (float)gs[j];
  if (src_norm)
    for (int64_t j = 0; j < num_cols * F; ++j) src_norm[j] = sqrt(gs2[j]);
  if (grad_edge)
    for (int64_t j = 0; j < nnz_total * H; ++j) grad_edge[j] = (float)ge[j];
  if (edge_norm && msg == MSG_SRC_MUL_EDGE)
    for (int64_t j = 0; j < nnz_total * H; ++j) edge_norm[j] = sqrt(ge2[j]);
  rc = 0;
done:
  free(fwd);
  free(arg);
  free(pos);
  free(gs);
  free(gs2);
  free(ge);
  free(ge2);
  return rc;
}

/*
 * Gradient of the edge softmax (with optional leaky ReLU) w.r.t. its input
 * scores.  With a_e the softmax of row v (head h) and G = dL/da:
 *   dL/ds'_e = a_e * (G_e - c),   c = sum_{p in row} a_p * G_p
 * (the Jacobian of softmax is diag(a) - a a^T), and through the leaky ReLU
 *   dL/ds_e = dL/ds'_e * (s_e > 0 ? 1 : slope)     (slope also at s_e = 0).
 * a is recomputed here from the scores in fp64 exactly as fgref_edge_softmax
 * defines it; the result is rounded to fp32 once.  scale (optional, indexed
 * like grad_scores) receives a_e * (|G_e| + sum_p a_p |G_p|) times the leaky
 * factor: the size of the terms the result is formed from.
 */
FGREF_EXPORT int fgref_edge_softmax_backward(int64_t num_rows, const int32_t* indptr,
                                             const int32_t* edge_ids, int64_t nnz_total,
                                             int64_t H, const float* scores,
                                             const float* grad_out, int apply_leaky_relu,
                                             float slope, const int64_t* rows, int64_t num_sel,
                                             float* grad_scores, double* scale,
                                             int num_threads) {
  if (H < 1 || num_rows < 0 || !indptr || !scores || !grad_out || !grad_scores) return -1;
  if (!rows && num_sel != num_rows) return -1;
  if (check_rows(rows, num_sel, num_rows)) return -1;
  set_threads(num_threads);
  int bad = 0;

#pragma omp parallel for schedule(dynamic, 64) reduction(| : bad)
  for (int64_t i = 0; i < num_sel; ++i) {
    const int64_t v = pick_row(rows, i);
    const int64_t p0 = indptr[v], p1 = indptr[v + 1];
    for (int64_t p = p0; p < p1; ++p) {
      const int64_t e = edge_ids ? edge_ids[p] : p;
      if (e < 0 || e >= nnz_total) bad |= 1;
    }
    if (bad) continue;
    for (int64_t h = 0; h < H; ++h) {
      double m = -INFINITY;
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        double s = scores[e * H + h];
        if (apply_leaky_relu && !(s > 0.0)) s = (double)slope * s;
        if (s > m) m = s;
      }
      double z = 0.0;
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        double s = scores[e * H + h];
        if (apply_leaky_relu && !(s > 0.0)) s = (double)slope * s;
        z += exp(s - m);
      }
      double c = 0.0, cabs = 0.0;
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        double s = scores[e * H + h];
        if (apply_leaky_relu && !(s > 0.0)) s = (double)slope * s;
        const double a = exp(s - m) / z;
        c += a * (double)grad_out[e * H + h];
        cabs += a * fabs((double)grad_out[e * H + h]);
      }
      for (int64_t p = p0; p < p1; ++p) {
        const int64_t e = edge_ids ? edge_ids[p] : p;
        const double s0 = scores[e * H + h];
        const double s = (apply_leaky_relu && !(s0 > 0.0)) ? (double)slope * s0 : s0;
        const double lf = (apply_leaky_relu && !(s0 > 0.0)) ? (double)slope : 1.0;
        const double a = exp(s - m) / z;
        const double g = grad_out[e * H + h];
        grad_scores[e * H + h] = (float)(a * (g - c) * lf);
        if (scale) scale[e * H + h] = a * (fabs(g) + cabs) * fabs(lf);
      }
    }
  }
  return bad ? -2 : 0;
}

/*
 * MLP aggregation (Fig. 1, with the message function of Fig. 3b): for every
 * stored edge (v <- u) with id e and every output feature i,
 *   m_e[i] = relu( sum_k (Xs[u, k] + Xd[v, k]) * W[k, i] ),  relu(t) = t > 0 ? t : 0
 * evaluated in fp64 (Xs [num_cols, d_in], Xd [num_rows, d_in], W [d_in, d_out]),
 * and the destination keeps the maximum message:
 *   out[v, i] = (float) max_e m_e[i],  arg[v, i] = the smallest edge id attaining it
 * (empty row -> out 0, arg -1).  scale (optional) receives
 * sum_k |Xs[u, k] + Xd[v, k]| * |W[k, i]| of the selected edge, the size of the
 * terms its message is formed from.
 */
FGREF_EXPORT int fgref_mlp_aggregate(int64_t num_rows, int64_t num_cols, const int32_t* indptr,
                                     const int32_t* indices, const int32_t* edge_ids,
                                     int64_t nnz_total, int64_t d_in, int64_t d_out,
                                     const float* xs, const float* xd, const float* w,
                                     const int64_t* rows, int64_t num_sel, float* out,
                                     int32_t* arg, double* scale, int num_threads) {
  if (d_in < 1 || d_out < 1 || num_rows < 0 || num_cols < 0 || !indptr || !xs || !xd || !w ||
      !out || !arg)
    return -1;
  if (!rows && num_sel != num_rows) return -1;
  if (check_rows(rows, num_sel, num_rows)) return -1;
  set_threads(num_threads);
  int bad = 0;

#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
  for (int64_t s = 0; s < num_sel; ++s) {
    const int64_t v = pick_row(rows, s);
    for (int64_t i = 0; i < d_out; ++i) {
      double best = 0.0, best_scale = 0.0;
      int32_t best_e = -1;
      for (int64_t p = indptr[v]; p < indptr[v + 1]; ++p) {
        const int64_t u = indices[p];
        const int64_t e = edge_ids ? edge_ids[p] : p;
        if (u < 0 || u >= num_cols || e < 0 || e >= nnz_total) { bad |= 1; continue; }
        double t = 0.0, sc = 0.0;
        for (int64_t k = 0; k < d_in; ++k) {
          const double h = (double)xs[u * d_in + k] + (double)xd[v * d_in + k];
          t += h * (double)w[k * d_out + i];
          sc += fabs(h) * fabs((double)w[k * d_out + i]);
        }
        const double m = t > 0.0 ? t : 0.0;
        if (best_e == -1 || m > best || (m == best && e < best_e)) {
          best = m;
          best_e = (int32_t)e;
          best_scale = sc;
        }
      }
      out[s * d_out + i] = best_e == -1 ? 0.0f : (float)best;
      arg[s * d_out + i] = best_e;
      if (scale) scale[s * d_out + i] = best_scale;
    }
  }
  return bad ? -2 : 0;
}

/*
 * Dense vertex transform of MLP aggregation (the vector-matrix product inside
 * the message function of Fig. 3b, applied to every vertex's features):
 *   Y[i, j] = sum_k X[i, k] * W[k, j]
 * with X [n, d_in] and W [d_in, d_out] row-major fp32, Y [n, d_out] fp64 (the
 * products and their sum in fp64, k in increasing order, no rounding to fp32).
 */
FGREF_EXPORT int fgref_dense_matmul(int64_t n, int64_t d_in, int64_t d_out, const float* x,
                                    const float* w, double* y, int num_threads) {
  if (n < 0 || d_in < 1 || d_out < 1 || (n > 0 && (!x || !w || !y))) return -1;
  set_threads(num_threads);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    for (int64_t j = 0; j < d_out; ++j) {
      double acc = 0.0;
      for (int64_t k = 0; k < d_in; ++k) acc += (double)x[i * d_in + k] * (double)w[k * d_out + j];
      y[i * d_out + j] = acc;
    }
  }
  return 0;
}

FGREF_EXPORT int fgref_max_threads(void) { return omp_get_max_threads(); }

/* Sets the OpenMP thread count used by later calls that pass num_threads = 0. */
FGREF_EXPORT void fgref_set_num_threads(int n) {
  if (n > 0) omp_set_num_threads(n);
}
