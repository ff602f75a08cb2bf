/*
 * AVQ-Attention forward pass: plain fp64 CPU oracle.
 *
 * TEST INFRASTRUCTURE ONLY. Only the tests, the smoke check and the CPU
 * baseline leg of the benchmark may load this library. The product path never
 * calls it, and it shares no code, header or table with the HIP kernels.
 *
 * Every function follows the paper's definitions directly, one term at a time,
 * in fp64 on inputs that were stored in bf16/fp32 and widened exactly:
 *   - assignment          Sec. 3.2 (nearest codeword, squared L2), Alg. 1 (tree:
 *                         nearest parent, then its children; a key moves only if
 *                         a child is strictly closer than its parent)
 *   - aggregates          Eq. (aggregates); parent rows cover the whole parent
 *                         cell, child rows the keys that moved (Alg. 1, App. C)
 *   - importance          Eq. (importance) with the exact denominator of the
 *                         parent pass (Eq. (vqflashattention)), empty codes
 *                         excluded (App. D)
 *   - top-P               Sec. 4.3 "child spawning": the P parents of largest
 *                         importance per query tile
 *   - refined output      Eq. (vqflashattention) over the parents, corrected by
 *                         Eq. (correcting_attention) for the children of every
 *                         selected parent; the parent logit is either recovered
 *                         from the children by Eq. (parent_recovery) (as the
 *                         fused kernel does) or taken directly (App. C form)
 *
 * Layouts (row-major, all contiguous):
 *   Q, K, V, Y        [BH][N][d]          bh = b*H + h, codebook head = bh % H
 *   Cp                [H][M0][d]
 *   Cc                [H][M0][Ch][d]
 *   Vbar              [BH][Mtot][d]        Mtot = M0*(1+Ch)
 *   counts            [BH][Mtot]           row M0 + p*Ch + c = child c of parent p
 *   importance        [BH][T][M0]          T = ceil(N / block_q)
 *   selection         [BH][T][P]           canonical order: w desc, index asc
 *
 * Readings where the paper is silent: the softmax scale is folded into Q
 * (logits are exactly Q.C); parent argmin ties go to the lowest index; a child
 * replaces the cached parent distance only when strictly smaller; the query
 * tile is block_q consecutive tokens and a ragged last tile uses its own rows;
 * top-P ties go to the lowest index.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

int avqo_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

void avqo_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* Squared Euclidean distance ||a - b||^2 (Sec. 3.2). */
static double sqdist(const double* a, const double* b, int d) {
  double s = 0.0;
  for (int e = 0; e < d; ++e) {
    double t = a[e] - b[e];
    s += t * t;
  }
  return s;
}

static double dot(const double* a, const double* b, int d) {
  double s = 0.0;
  for (int e = 0; e < d; ++e) s += a[e] * b[e];
  return s;
}

/*
 * Tree assignment (Sec. 3.2 assignment; Alg. 1 parent and child loops).
 * For key j: p* = lowest index attaining min_a ||K_j - Cp_a||^2; then
 * c* = lowest child index attaining min_c ||K_j - Cc_{p*,c}||^2; the key moves
 * to child c* iff that distance is strictly below the parent distance.
 * Outputs parent_idx[j] = p*, code_idx[j] = p* (stays) or M0 + p*Ch + c*.
 * Optional certification outputs (nullable), all [BH][N]:
 *   d_parent     distance to p*
 *   d_parent2    second-smallest parent distance (+inf if M0 == 1)
 *   d_child      distance to c*
 *   d_child2     second-smallest child distance (+inf if Ch == 1)
 */
void avqo_assign(int BH, int H, int N, int d, int M0, int Ch,
                 const double* K, const double* Cp, const double* Cc,
                 int32_t* parent_idx, int32_t* code_idx,
                 double* d_parent, double* d_parent2,
                 double* d_child, double* d_child2) {
  long long total = (long long)BH * N;
#pragma omp parallel for schedule(static)
  for (long long t = 0; t < total; ++t) {
    int bh = (int)(t / N);
    int h = bh % H;
    const double* k = K + t * d;
    int best = 0;
    double dbest = INFINITY, dsecond = INFINITY;
    for (int a = 0; a < M0; ++a) {
      double dist = sqdist(k, Cp + ((long long)h * M0 + a) * d, d);
      if (dist < dbest) {
        dsecond = dbest;
        dbest = dist;
        best = a;
      } else if (dist < dsecond) {
        dsecond = dist;
      }
    }
    int cbest = 0;
    double dc = INFINITY, dc2 = INFINITY;
    for (int c = 0; c < Ch; ++c) {
      double dist = sqdist(k, Cc + (((long long)h * M0 + best) * Ch + c) * d, d);
      if (dist < dc) {
        dc2 = dc;
        dc = dist;
        cbest = c;
      } else if (dist < dc2) {
        dc2 = dist;
      }
    }
    parent_idx[t] = best;
    code_idx[t] = (dc < dbest) ? (M0 + best * Ch + cbest) : best;
    if (d_parent) d_parent[t] = dbest;
    if (d_parent2) d_parent2[t] = dsecond;
    if (d_child) d_child[t] = dc;
    if (d_child2) d_child2[t] = dc2;
  }
}

/*
 * Aggregates, Eq. (aggregates): n_a = number of keys with code a and
 * Vbar_a = sum of their values. Parent rows a < M0 collect every key whose
 * nearest parent is a (Alg. 1 adds to the parent unconditionally); child rows
 * collect only the keys that moved to that child.
 */
void avqo_aggregate(int BH, int N, int d, int M0, int Ch, const double* V,
                    const int32_t* parent_idx, const int32_t* code_idx,
                    double* Vbar, int64_t* counts) {
  int Mtot = M0 * (1 + Ch);
#pragma omp parallel for schedule(static)
  for (int bh = 0; bh < BH; ++bh) {
    double* vb = Vbar + (long long)bh * Mtot * d;
    int64_t* n = counts + (long long)bh * Mtot;
    memset(vb, 0, sizeof(double) * (size_t)Mtot * d);
    memset(n, 0, sizeof(int64_t) * (size_t)Mtot);
    for (int j = 0; j < N; ++j) {
      long long t = (long long)bh * N + j;
      const double* v = V + t * d;
      int p = parent_idx[t];
      n[p] += 1;
      for (int e = 0; e < d; ++e) vb[(long long)p * d + e] += v[e];
      int code = code_idx[t];
      if (code >= M0) {
        n[code] += 1;
        for (int e = 0; e < d; ++e) vb[(long long)code * d + e] += v[e];
      }
    }
  }
}

/*
 * Per-tile parent importance, Eq. (importance):
 *   w_a(I) = sum_{i in I} n_a exp(S_ia) / Zbar_i,  Zbar_i = sum_a' n_a' exp(S_ia'),
 * with S_ia = Q_i . Cp_a over non-empty parents only (empty parents get w = 0,
 * App. D). The max shift mu_i cancels and only keeps exp() in range.
 * tile_mask (nullable, [BH][T]) restricts the work to tiles with a non-zero
 * entry; other rows of w are left untouched.
 */
void avqo_importance(int BH, int H, int N, int d, int M0, int Ch, int block_q,
                     const double* Q, const double* Cp, const int64_t* counts,
                     const uint8_t* tile_mask, double* w) {
  int T = (N + block_q - 1) / block_q;
  int Mtot = M0 * (1 + Ch);
  long long total = (long long)BH * T;
#pragma omp parallel for schedule(dynamic, 1)
  for (long long bt = 0; bt < total; ++bt) {
    if (tile_mask && !tile_mask[bt]) continue;
    int bh = (int)(bt / T), t = (int)(bt % T), h = bh % H;
    const int64_t* n = counts + (long long)bh * Mtot;
    double* wt = w + bt * M0;
    double* S = (double*)malloc(sizeof(double) * M0);
    for (int a = 0; a < M0; ++a) wt[a] = 0.0;
    int i_end = (t + 1) * block_q < N ? (t + 1) * block_q : N;
    for (int i = t * block_q; i < i_end; ++i) {
      const double* q = Q + ((long long)bh * N + i) * d;
      double mu = -INFINITY;
      for (int a = 0; a < M0; ++a) {
        S[a] = dot(q, Cp + ((long long)h * M0 + a) * d, d);
        if (n[a] > 0 && S[a] > mu) mu = S[a];
      }
      double Z = 0.0;
      for (int a = 0; a < M0; ++a)
        if (n[a] > 0) Z += (double)n[a] * exp(S[a] - mu);
      for (int a = 0; a < M0; ++a)
        if (n[a] > 0) wt[a] += (double)n[a] * exp(S[a] - mu) / Z;
    }
    free(S);
  }
}

/*
 * Importance with tiled codewords (App. B, Eq. (aproxdenom) and
 * Eq. (codewordimportance)): the parents are visited in consecutive tiles of
 * tile_c. After tile J, the partial denominator of query i (the sum of
 * n_a exp(S_ia) over the non-empty parents of tiles up to J) is scaled by
 * N / N_seen(J), N_seen(J) being the number of keys in the parents of those
 * tiles, and the importance of every parent a of tile J is
 * w_a += n_a exp(S_ia) / Ztilde_i(J). For the last tile N_seen = N and the
 * result is Eq. (importance); a tile with N_seen = 0 holds only empty parents,
 * which get w = 0. The shift mu_i cancels in each ratio.
 */
void avqo_importance_tiled(int BH, int H, int N, int d, int M0, int Ch, int block_q, int tile_c,
                           const double* Q, const double* Cp, const int64_t* counts,
                           const uint8_t* tile_mask, double* w) {
  int T = (N + block_q - 1) / block_q;
  int Mtot = M0 * (1 + Ch);
  long long total = (long long)BH * T;
#pragma omp parallel for schedule(dynamic, 1)
  for (long long bt = 0; bt < total; ++bt) {
    if (tile_mask && !tile_mask[bt]) continue;
    int bh = (int)(bt / T), t = (int)(bt % T), h = bh % H;
    const int64_t* n = counts + (long long)bh * Mtot;
    double* wt = w + bt * M0;
    double* S = (double*)malloc(sizeof(double) * M0);
    for (int a = 0; a < M0; ++a) wt[a] = 0.0;
    int i_end = (t + 1) * block_q < N ? (t + 1) * block_q : N;
    for (int i = t * block_q; i < i_end; ++i) {
      const double* q = Q + ((long long)bh * N + i) * d;
      double mu = -INFINITY;
      for (int a = 0; a < M0; ++a) {
        S[a] = dot(q, Cp + ((long long)h * M0 + a) * d, d);
        if (n[a] > 0 && S[a] > mu) mu = S[a];
      }
      double zsum = 0.0;
      long long seen = 0;
      for (int a0 = 0; a0 < M0; a0 += tile_c) {
        int a1 = a0 + tile_c < M0 ? a0 + tile_c : M0;
        for (int a = a0; a < a1; ++a) {
          seen += n[a];
          if (n[a] > 0) zsum += (double)n[a] * exp(S[a] - mu);
        }
        if (seen == 0) continue;
        double zt = (double)N / (double)seen * zsum;
        for (int a = a0; a < a1; ++a)
          if (n[a] > 0) wt[a] += (double)n[a] * exp(S[a] - mu) / zt;
      }
    }
    free(S);
  }
}

/*
 * Top-P (Sec. 4.3, child spawning): for every row of w (length M0), the P
 * parents of largest importance, listed in the canonical order
 * (importance descending, index ascending on equal importance).
 * Selection by repeated maximum: each step takes the best parent not yet taken.
 */
void avqo_topp(long long rows, int M0, int P, const double* w, const uint8_t* row_mask,
               int32_t* sel) {
#pragma omp parallel for schedule(static)
  for (long long r = 0; r < rows; ++r) {
    if (row_mask && !row_mask[r]) continue;
    const double* wr = w + r * M0;
    uint8_t* taken = (uint8_t*)calloc((size_t)M0, 1);
    for (int k = 0; k < P; ++k) {
      int best = -1;
      for (int a = 0; a < M0; ++a) {
        if (taken[a]) continue;
        if (best < 0 || wr[a] > wr[best]) best = a;
      }
      taken[best] = 1;
      sel[r * P + k] = best;
    }
    free(taken);
  }
}

/*
 * Refined output for every query i of tile I (Eq. (vqflashattention) over the
 * parents, then Eq. (correcting_attention) for the children of each selected
 * parent, App. C):
 *   X_i = sum_{a: n_a>0} e^{S_ia} Vbar_a
 *       + sum_{p in S_I} sum_{c: n_pc>0} (e^{T_ipc} - e^{R_ip}) Vbar_pc
 *   Z_i = the same with n in place of Vbar,       Y_i = X_i / Z_i
 * with T_ipc = Q_i . Cc_pc and R_ip the parent logit: recovered as the mean of
 * all Ch child logits, Eq. (parent_recovery) (recovered != 0), or the direct
 * Q_i . Cp_p (recovered == 0). Every exponent is shifted by one finite mu_i
 * (max over the non-empty parent and child logits), which cancels in X/Z.
 * Z_out (nullable, [BH][N]) receives Z_i / sum_{a: n_a>0} n_a e^{S_ia}, the
 * refined denominator relative to the parent-only one, so that the tests can
 * check its sign and size.
 */
void avqo_output(int BH, int H, int N, int d, int M0, int Ch, int P, int block_q,
                 const double* Q, const double* Cp, const double* Cc,
                 const double* Vbar, const int64_t* counts, const int32_t* sel,
                 int recovered, const uint8_t* tile_mask, double* Y, double* Z_out) {
  int T = (N + block_q - 1) / block_q;
  int Mtot = M0 * (1 + Ch);
  long long total = (long long)BH * T;
#pragma omp parallel for schedule(dynamic, 1)
  for (long long bt = 0; bt < total; ++bt) {
    if (tile_mask && !tile_mask[bt]) continue;
    int bh = (int)(bt / T), t = (int)(bt % T), h = bh % H;
    const int64_t* n = counts + (long long)bh * Mtot;
    const double* vb = Vbar + (long long)bh * Mtot * d;
    const int32_t* s = sel + bt * P;
    double* S = (double*)malloc(sizeof(double) * M0);
    double* Tc = (double*)malloc(sizeof(double) * (P > 0 ? P : 1) * Ch);
    double* R = (double*)malloc(sizeof(double) * (P > 0 ? P : 1));
    double* X = (double*)malloc(sizeof(double) * d);
    int i_end = (t + 1) * block_q < N ? (t + 1) * block_q : N;
    for (int i = t * block_q; i < i_end; ++i) {
      const double* q = Q + ((long long)bh * N + i) * d;
      double mu = -INFINITY;
      for (int a = 0; a < M0; ++a) {
        S[a] = dot(q, Cp + ((long long)h * M0 + a) * d, d);
        if (n[a] > 0 && S[a] > mu) mu = S[a];
      }
      for (int k = 0; k < P; ++k) {
        int p = s[k];
        double mean = 0.0;
        for (int c = 0; c < Ch; ++c) {
          double v = dot(q, Cc + (((long long)h * M0 + p) * Ch + c) * d, d);
          Tc[k * Ch + c] = v;
          mean += v;
          if (n[M0 + p * Ch + c] > 0 && v > mu) mu = v;
        }
        R[k] = recovered ? mean / Ch : S[p];
      }
      double Z = 0.0, Zp = 0.0;
      for (int e = 0; e < d; ++e) X[e] = 0.0;
      for (int a = 0; a < M0; ++a) {
        if (n[a] == 0) continue;
        double A = exp(S[a] - mu);
        Z += A * (double)n[a];
        Zp += A * (double)n[a];
        for (int e = 0; e < d; ++e) X[e] += A * vb[(long long)a * d + e];
      }
      for (int k = 0; k < P; ++k) {
        int p = s[k];
        double Ap = exp(R[k] - mu);
        for (int c = 0; c < Ch; ++c) {
          int code = M0 + p * Ch + c;
          if (n[code] == 0) continue;
          double dA = exp(Tc[k * Ch + c] - mu) - Ap;
          Z += dA * (double)n[code];
          for (int e = 0; e < d; ++e) X[e] += dA * vb[(long long)code * d + e];
        }
      }
      double* y = Y + ((long long)bh * N + i) * d;
      for (int e = 0; e < d; ++e) y[e] = X[e] / Z;
      if (Z_out) Z_out[(long long)bh * N + i] = Z / Zp;
    }
    free(S);
    free(Tc);
    free(R);
    free(X);
  }
}

/*
 * Codebook update by exponential moving averages with the parent-child
 * constraint (App. A). For every head h and code x (parents and children),
 * the batch statistics are the key sums and counts of that code over all
 * batch entries b (parent rows cover the whole parent cell, as the
 * aggregates of Eq. (aggregates) do):
 *   S_x <- lambda S_x + (1 - lambda) sum_b sums[b][h][x],
 *   N_x <- lambda N_x + (1 - lambda) sum_b counts[b][h][x].
 * Parents take the unconstrained mean, C_p = S_p / N_p. The children of p,
 * with unconstrained means M_c = S_c / N_c, are projected onto the constraint
 * (mean of the children = C_p) by the mass-weighted least-squares solution
 * Eq. (child_constraint_solve):
 *   delta = sum_c M_c - Ch C_p,  sigma = sum_c 1 / N_c,
 *   C_pc = M_c - delta / (N_c sigma).
 * S [H][Mtot][d] and Nema [H][Mtot] are updated in place; Cp_out [H][M0][d]
 * and Cc_out [H][M0][Ch][d] receive the new codewords.
 */
void avqo_codebook_update(int B, int H, int d, int M0, int Ch, double lambda,
                          const double* sums, const int64_t* counts, double* S, double* Nema,
                          double* Cp_out, double* Cc_out) {
  int Mtot = M0 * (1 + Ch);
#pragma omp parallel for schedule(static)
  for (int h = 0; h < H; ++h) {
    for (int x = 0; x < Mtot; ++x) {
      double n = 0.0;
      for (int b = 0; b < B; ++b) n += (double)counts[((long long)b * H + h) * Mtot + x];
      long long r = (long long)h * Mtot + x;
      Nema[r] = lambda * Nema[r] + (1.0 - lambda) * n;
      for (int e = 0; e < d; ++e) {
        double sx = 0.0;
        for (int b = 0; b < B; ++b) sx += sums[(((long long)b * H + h) * Mtot + x) * d + e];
        S[r * d + e] = lambda * S[r * d + e] + (1.0 - lambda) * sx;
      }
    }
    for (int p = 0; p < M0; ++p) {
      long long rp = (long long)h * Mtot + p;
      double* cp = Cp_out + ((long long)h * M0 + p) * d;
      for (int e = 0; e < d; ++e) cp[e] = S[rp * d + e] / Nema[rp];
      if (Ch == 0) continue;
      double sigma = 0.0;
      for (int c = 0; c < Ch; ++c) sigma += 1.0 / Nema[(long long)h * Mtot + M0 + p * Ch + c];
      for (int e = 0; e < d; ++e) {
        double delta = -(double)Ch * cp[e];
        for (int c = 0; c < Ch; ++c) {
          long long rc = (long long)h * Mtot + M0 + p * Ch + c;
          delta += S[rc * d + e] / Nema[rc];
        }
        for (int c = 0; c < Ch; ++c) {
          long long rc = (long long)h * Mtot + M0 + p * Ch + c;
          Cc_out[(((long long)h * M0 + p) * Ch + c) * d + e] =
              S[rc * d + e] / Nema[rc] - delta / (Nema[rc] * sigma);
        }
      }
    }
  }
}
