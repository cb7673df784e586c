/*
 * Gefen oracle: a plain, slow, float64 CPU definition of what the Gefen optimizer
 * computes ("Gefen: Optimized Stochastic Optimizer", arXiv 2606.13894).
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may call, link or load this
 * file; it exists so that tests, the smoke check and the benchmark's CPU-baseline leg
 * can check the HIP library against an independent definition. It shares no code,
 * header, table or constant with the HIP sources.
 *
 * Every routine is a sequential loop in float64 with no blocking, fusion or
 * reordering beyond what the paper states. Gradients arrive as fp32 or bf16 bits and
 * are widened exactly to float64. Build with -ffp-contract=off and without fast-math.
 *
 * Readings of the paper where it is silent or ambiguous (each one is listed in the
 * design notes of the repository as well):
 *   R1  eps inside log(g^2 + eps) of the partition score is a parameter (eps_part).
 *   R2  S(n) (a single block, 0/0 in the score equation) is defined as 0.
 *   R3  the neighbours of a candidate period are the adjacent entries of the full
 *       sorted divisor list, 1 and n included.
 *   R4  argmax ties among candidate periods go to the smallest period.
 *   R5  histogram bin of x in [-1, 1] over NB bins is floor((x + 1) * NB / 2),
 *       clamped to NB - 1 (so x = +1 lands in the last bin).
 *   R6  DP argmin ties go to the smallest left boundary.
 *   R7  fewer non-empty bins (b) than codebook entries (k): the DP is solved with
 *       max(b, 2) entries when b >= 2 and the codebook is padded with +1; with b < 2
 *       the codebook is {-1, +1, +1, ...}. Status 1 ("degenerate") is returned.
 *   R8  nearest codebook entry: argmin_j |x - c_j|, ties to the smaller j; a block
 *       whose new scale is 0 stores code 0 for every element.
 *   R9  the bias-corrected momentum uses the unquantized m_t of the same step.
 *   R10 per-block second moment uses the mean of g^2 over the block's elements.
 *   R11 Gefen-Muon: the quantized buffer is Muon's momentum (no second moment); the
 *       matrix that is orthogonalised is formed from the unquantized momentum of the
 *       same step (as R9), with Muon's Nesterov interpolation when enabled.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Gradient element i as float64. dtype 0: fp32; dtype 1: bf16 (upper half of fp32). */
static double grad_at(const void* g, int32_t dtype, int64_t i)
{
    if (dtype == 0) {
        return (double)((const float*)g)[i];
    }
    uint32_t bits = ((uint32_t)((const uint16_t*)g)[i]) << 16;
    float f;
    memcpy(&f, &bits, sizeof f);
    return (double)f;
}

/* ------------------------------------------------------------------------------
 * Divisors of n in increasing order (Alg. 2, the candidate period list P).
 * Returns the number of divisors; writes at most `cap` of them.
 * ---------------------------------------------------------------------------- */
int64_t oracle_divisors(int64_t n, int64_t* out, int64_t cap)
{
    if (n < 1) return 0;
    int64_t small_cnt = 0, large_cnt = 0, room = 64;
    /* small divisors ascending, large ones descending; merged at the end */
    int64_t* small = (int64_t*)malloc(sizeof(int64_t) * (size_t)room);
    int64_t* large = (int64_t*)malloc(sizeof(int64_t) * (size_t)room);
    for (int64_t d = 1; d <= n / d; ++d) {
        if (n % d == 0) {
            if (small_cnt == room) {
                room *= 2;
                small = (int64_t*)realloc(small, sizeof(int64_t) * (size_t)room);
                large = (int64_t*)realloc(large, sizeof(int64_t) * (size_t)room);
            }
            small[small_cnt++] = d;
            if (d != n / d) large[large_cnt++] = n / d;
        }
    }
    int64_t total = small_cnt + large_cnt, w = 0;
    for (int64_t i = 0; i < small_cnt; ++i) { if (w < cap) out[w] = small[i]; ++w; }
    for (int64_t i = large_cnt - 1; i >= 0; --i) { if (w < cap) out[w] = large[i]; ++w; }
    free(small);
    free(large);
    return total;
}

/* ------------------------------------------------------------------------------
 * Automatic Block Partitioning (Sec. 5.1, Alg. 2 and the partition-score equation).
 *
 *   z_j   = log(g_j^2 + eps)
 *   mu_i  = (1/p) * sum of z over the i-th consecutive block of p elements
 *   S(p)  = mean over i of |mu_{i+1} - mu_i|      (S(n) = 0, reading R2)
 *   keep p with 1 < p < n whose S is strictly larger than both neighbours' (R3),
 *   return the kept p with the largest S (R4), or 1 if none is kept.
 *
 * divs/scores receive the divisor list and S values (at most cap entries).
 * Returns 0 on success, -1 if cap is too small or n < 1.
 * ---------------------------------------------------------------------------- */
int oracle_partition(const void* g, int32_t dtype, int64_t n, double eps,
                     int64_t* divs, double* scores, int64_t cap,
                     int64_t* n_div_out, int64_t* period_out)
{
    if (n < 1) return -1;
    int64_t nd = oracle_divisors(n, divs, cap);
    *n_div_out = nd;
    if (nd > cap) return -1;

    double* z = (double*)malloc(sizeof(double) * (size_t)n);
    for (int64_t j = 0; j < n; ++j) {
        double gj = grad_at(g, dtype, j);
        z[j] = log(gj * gj + eps);
    }

    for (int64_t d = 0; d < nd; ++d) {
        int64_t p = divs[d];
        int64_t nb = n / p;
        if (nb < 2) {                      /* p == n: a single block (R2) */
            scores[d] = 0.0;
            continue;
        }
        double contrast = 0.0;
        double prev_mu = 0.0;
        for (int64_t i = 0; i < nb; ++i) {
            double sum = 0.0;
            for (int64_t j = i * p; j < (i + 1) * p; ++j) sum += z[j];
            double mu = sum / (double)p;
            if (i > 0) contrast += fabs(mu - prev_mu);
            prev_mu = mu;
        }
        scores[d] = contrast / (double)(nb - 1);
    }
    free(z);

    /* strict local maxima among 1 < p < n, then argmax (first one on ties) */
    int64_t best = 1;
    double best_s = 0.0;
    int have = 0;
    for (int64_t d = 1; d + 1 < nd; ++d) {
        double s = scores[d];
        if (s > scores[d - 1] && s > scores[d + 1]) {
            if (!have || s > best_s) {
                best = divs[d];
                best_s = s;
                have = 1;
            }
        }
    }
    *period_out = best;
    return 0;
}

/* ------------------------------------------------------------------------------
 * Block-normalised gradient histogram (Alg. 3, first loop).
 * Blocks are [offs[b], offs[b+1]). A block whose absolute maximum is 0 is skipped.
 * Each element x = g / max|g_block| is counted into bin floor((x + 1) * NB / 2),
 * clamped to NB - 1 (reading R5). Counts are added to hist (caller clears it).
 * ---------------------------------------------------------------------------- */
void oracle_histogram_blocks(const void* g, int32_t dtype, const int64_t* offs,
                             int64_t nblocks, int32_t nbins, uint64_t* hist)
{
    double half = (double)nbins / 2.0;
    for (int64_t b = 0; b < nblocks; ++b) {
        double a = 0.0;
        for (int64_t i = offs[b]; i < offs[b + 1]; ++i) {
            double x = fabs(grad_at(g, dtype, i));
            if (x > a) a = x;
        }
        if (a == 0.0) continue;
        for (int64_t i = offs[b]; i < offs[b + 1]; ++i) {
            double x = grad_at(g, dtype, i) / a;
            int64_t bin = (int64_t)floor((x + 1.0) * half);
            if (bin > nbins - 1) bin = nbins - 1;
            if (bin < 0) bin = 0;
            hist[bin] += 1;
        }
    }
}

/* Same with uniform blocks of p elements over a tensor of n elements (p divides n). */
void oracle_histogram_uniform(const void* g, int32_t dtype, int64_t n, int64_t p,
                              int32_t nbins, uint64_t* hist)
{
    int64_t nb = n / p;
    int64_t offs[2];
    for (int64_t b = 0; b < nb; ++b) {
        offs[0] = b * p;
        offs[1] = (b + 1) * p;
        oracle_histogram_blocks((const char*)g, dtype, offs, 1, nbins, hist);
    }
}

/* ------------------------------------------------------------------------------
 * Exact histogram DP codebook (Alg. 3 and App. D).
 *
 * Non-empty bins i (in increasing order) with centre m_i = -1 + (i + 1/2) * (2/NB)
 * and count c_i. Prefix sums Z0, Z1, Z2 of c, c*m, c*m*m. For bins [l, r]
 * (1-based, inclusive) with S_q = Z_q[r] - Z_q[l-1]:
 *   entry 1 (centre -1) and entry k (centre +1): C = S2 - 2 a S1 + a^2 S0
 *   entries 2..k-1:                              C = S2 - S1^2 / S0
 * D[0][0] = 0, all other entries +inf;
 * D[r][j] = min over l in [j, r] of D[l-1][j-1] + C(l, r, j), ties to the smallest l.
 * Backtracking the stored l recovers the intervals; entry j is -1, +1 or S1/S0.
 *
 * Outputs: codebook[k] (sorted), *cost = D[b][k], bounds[k] = first bin (1-based,
 * compacted order) of each interval. Returns 0, 1 for the degenerate case (R7),
 * or -1 for invalid arguments (k < 2).
 * ---------------------------------------------------------------------------- */
static double interval_cost(const double* Z0, const double* Z1, const double* Z2,
                            int64_t l, int64_t r, int32_t j, int32_t k)
{
    double S0 = Z0[r] - Z0[l - 1];
    double S1 = Z1[r] - Z1[l - 1];
    double S2 = Z2[r] - Z2[l - 1];
    if (j == 1 || j == k) {
        double a = (j == 1) ? -1.0 : 1.0;
        return S2 - 2.0 * a * S1 + a * a * S0;
    }
    return S2 - S1 * S1 / S0;
}

static void solve_dp(const double* Z0, const double* Z1, const double* Z2, int64_t b,
                     int32_t k, double* codebook, double* cost, int32_t* bounds)
{
    /* D and split are (b + 1) x (k + 1), row-major by r */
    size_t stride = (size_t)k + 1;
    double* D = (double*)malloc(sizeof(double) * (size_t)(b + 1) * stride);
    int32_t* split = (int32_t*)malloc(sizeof(int32_t) * (size_t)(b + 1) * stride);
    for (size_t i = 0; i < (size_t)(b + 1) * stride; ++i) {
        D[i] = INFINITY;
        split[i] = 0;
    }
    D[0] = 0.0;
    for (int32_t j = 1; j <= k; ++j) {
        for (int64_t r = j; r <= b; ++r) {
            double best = INFINITY;
            int64_t arg = 0;
            for (int64_t l = j; l <= r; ++l) {
                double cand = D[(size_t)(l - 1) * stride + (size_t)(j - 1)] +
                              interval_cost(Z0, Z1, Z2, l, r, j, k);
                if (cand < best) {
                    best = cand;
                    arg = l;
                }
            }
            D[(size_t)r * stride + (size_t)j] = best;
            split[(size_t)r * stride + (size_t)j] = (int32_t)arg;
        }
    }
    *cost = D[(size_t)b * stride + (size_t)k];
    int64_t r = b;
    for (int32_t j = k; j >= 1; --j) {
        int64_t l = split[(size_t)r * stride + (size_t)j];
        bounds[j - 1] = (int32_t)l;
        if (j == 1) {
            codebook[j - 1] = -1.0;
        } else if (j == k) {
            codebook[j - 1] = 1.0;
        } else {
            double S0 = Z0[r] - Z0[l - 1];
            double S1 = Z1[r] - Z1[l - 1];
            codebook[j - 1] = S1 / S0;
        }
        r = l - 1;
    }
    free(D);
    free(split);
}

int oracle_dp_codebook(const uint64_t* hist, int32_t nbins, int32_t k,
                       double* codebook, double* cost, int32_t* bounds)
{
    if (k < 2 || nbins < 1) return -1;
    double w = 2.0 / (double)nbins;
    int64_t b = 0;
    for (int32_t i = 0; i < nbins; ++i) if (hist[i] > 0) ++b;

    double* Z0 = (double*)malloc(sizeof(double) * (size_t)(b + 1));
    double* Z1 = (double*)malloc(sizeof(double) * (size_t)(b + 1));
    double* Z2 = (double*)malloc(sizeof(double) * (size_t)(b + 1));
    double* centres = (double*)malloc(sizeof(double) * (size_t)(b + 1));
    double* counts = (double*)malloc(sizeof(double) * (size_t)(b + 1));
    Z0[0] = Z1[0] = Z2[0] = 0.0;
    int64_t r = 0;
    for (int32_t i = 0; i < nbins; ++i) {
        if (hist[i] == 0) continue;
        double c = (double)hist[i];
        double m = -1.0 + ((double)i + 0.5) * w;
        ++r;
        centres[r] = m;
        counts[r] = c;
        Z0[r] = Z0[r - 1] + c;
        Z1[r] = Z1[r - 1] + c * m;
        Z2[r] = Z2[r - 1] + c * m * m;
    }

    int status = 0;
    for (int32_t j = 0; j < k; ++j) bounds[j] = 0;
    if (b >= k) {
        solve_dp(Z0, Z1, Z2, b, k, codebook, cost, bounds);
    } else {
        status = 1;
        if (b >= 2) {
            int32_t keff = (int32_t)b;
            solve_dp(Z0, Z1, Z2, b, keff, codebook, cost, bounds);
            for (int32_t j = keff; j < k; ++j) codebook[j] = 1.0;
        } else {
            codebook[0] = -1.0;
            for (int32_t j = 1; j < k; ++j) codebook[j] = 1.0;
            double e = 0.0;
            for (int64_t i = 1; i <= b; ++i) {
                double dl = centres[i] + 1.0, dr = 1.0 - centres[i];
                double d2 = (dl * dl < dr * dr) ? dl * dl : dr * dr;
                e += counts[i] * d2;
            }
            *cost = e;
        }
    }
    free(Z0);
    free(Z1);
    free(Z2);
    free(centres);
    free(counts);
    return status;
}

/* ------------------------------------------------------------------------------
 * One Gefen step (Alg. 1, the loop body) over blocks [offs[b], offs[b+1]).
 *
 *   m_i   = beta1 * (c_dec[q_i] * s) + (1 - beta1) * g_i          dequantize + EMA
 *   s'    = max_i |m_i|;  q'_i = nearest(c_enc, m_i / s')          requantize (R8)
 *   mhat  = m_i / (1 - beta1^t)                                    (R9)
 *   v'    = beta2 * v + (1 - beta2) * mean_i(g_i^2)                shared moment (R10)
 *   vhat  = v' / (1 - beta2^t)
 *   theta = theta - lr * (mhat / (sqrt(vhat) + eps) + wd * theta)
 *
 * theta, s, v are float64 arrays updated in place; codes are uint8 updated in place.
 * With quantize == 0 the momentum is kept unquantized in m_full (one float64 per
 * element) instead of codes and scales; this is the oracle-only no-quantization switch.
 * ---------------------------------------------------------------------------- */
void oracle_step_blocks(double* theta, const void* g, int32_t dtype, uint8_t* codes,
                        double* s, double* v, const int64_t* offs, int64_t nblocks,
                        const double* cb_dec, const double* cb_enc, int32_t k,
                        double lr, double beta1, double beta2, double eps, double wd,
                        int64_t t, int32_t quantize, double* m_full, double* m_out)
{
    double bc1 = 1.0 - pow(beta1, (double)t);
    double bc2 = 1.0 - pow(beta2, (double)t);
    for (int64_t b = 0; b < nblocks; ++b) {
        int64_t lo = offs[b], hi = offs[b + 1];
        int64_t len = hi - lo;
        if (len <= 0) continue;
        double* m = (double*)malloc(sizeof(double) * (size_t)len);
        double sumsq = 0.0;
        double smax = 0.0;
        for (int64_t i = lo; i < hi; ++i) {
            double gi = grad_at(g, dtype, i);
            double prev = quantize ? cb_dec[codes[i]] * s[b] : m_full[i];
            double mi = beta1 * prev + (1.0 - beta1) * gi;
            m[i - lo] = mi;
            sumsq += gi * gi;
            if (fabs(mi) > smax) smax = fabs(mi);
        }
        double vn = beta2 * v[b] + (1.0 - beta2) * (sumsq / (double)len);
        double vhat = vn / bc2;
        double denom = sqrt(vhat) + eps;
        for (int64_t i = lo; i < hi; ++i) {
            double mi = m[i - lo];
            if (m_out) m_out[i] = mi;
            if (quantize) {
                int32_t q = 0;
                if (smax > 0.0) {
                    double x = mi / smax;
                    double bd = fabs(x - cb_enc[0]);
                    for (int32_t j = 1; j < k; ++j) {
                        double d = fabs(x - cb_enc[j]);
                        if (d < bd) {
                            bd = d;
                            q = j;
                        }
                    }
                }
                codes[i] = (uint8_t)q;
            } else {
                m_full[i] = mi;
            }
            double mhat = mi / bc1;
            theta[i] = theta[i] - lr * (mhat / denom + wd * theta[i]);
        }
        s[b] = smax;
        v[b] = vn;
        free(m);
    }
}

/* Uniform blocks of p elements over n elements (p divides n). */
void oracle_step_uniform(double* theta, const void* g, int32_t dtype, uint8_t* codes,
                         double* s, double* v, int64_t n, int64_t p,
                         const double* cb_dec, const double* cb_enc, int32_t k,
                         double lr, double beta1, double beta2, double eps, double wd,
                         int64_t t, int32_t quantize, double* m_full, double* m_out)
{
    int64_t nb = n / p;
    int64_t* offs = (int64_t*)malloc(sizeof(int64_t) * (size_t)(nb + 1));
    for (int64_t b = 0; b <= nb; ++b) offs[b] = b * p;
    oracle_step_blocks(theta, g, dtype, codes, s, v, offs, nb, cb_dec, cb_enc, k, lr,
                       beta1, beta2, eps, wd, t, quantize, m_full, m_out);
    free(offs);
}

/* ------------------------------------------------------------------------------
 * Gefen-Muon momentum codec (appendix "Gefen-Muon"): Muon keeps one momentum buffer
 * per matrix and orthogonalises it; Gefen-Muon stores that buffer in Gefen's form
 * (per-element codes, one scale per block) and leaves the orthogonalisation as in
 * Muon. Over blocks [offs[b], offs[b+1]):
 *
 *   m_i  = mu * (c_dec[q_i] * s) + (1 - mu) * g_i        Muon's momentum EMA, decoded
 *   s'   = max_i |m_i|;  q'_i = nearest(c_enc, m_i / s')  requantize (R8)
 *   u_i  = nesterov ? (1 - mu) * g_i + mu * m_i : m_i     the matrix handed to the
 *                                                         orthogonalisation (R11)
 *
 * The Nesterov form follows Muon's: the update interpolates from the gradient towards
 * the new momentum by mu. Codes and s are updated in place; u is written (float64).
 * ---------------------------------------------------------------------------- */
void oracle_muon_codec_blocks(const void* g, int32_t dtype, uint8_t* codes, double* s,
                              const int64_t* offs, int64_t nblocks, const double* cb_dec,
                              const double* cb_enc, int32_t k, double mu, int32_t nesterov,
                              double* u)
{
    for (int64_t b = 0; b < nblocks; ++b) {
        int64_t lo = offs[b], hi = offs[b + 1];
        if (hi <= lo) continue;
        double smax = 0.0;
        for (int64_t i = lo; i < hi; ++i) {
            double gi = grad_at(g, dtype, i);
            double mi = mu * (cb_dec[codes[i]] * s[b]) + (1.0 - mu) * gi;
            u[i] = mi;
            if (fabs(mi) > smax) smax = fabs(mi);
        }
        for (int64_t i = lo; i < hi; ++i) {
            double mi = u[i];
            int32_t q = 0;
            if (smax > 0.0) {
                double x = mi / smax;
                double bd = fabs(x - cb_enc[0]);
                for (int32_t j = 1; j < k; ++j) {
                    double d = fabs(x - cb_enc[j]);
                    if (d < bd) {
                        bd = d;
                        q = j;
                    }
                }
            }
            codes[i] = (uint8_t)q;
            if (nesterov) u[i] = (1.0 - mu) * grad_at(g, dtype, i) + mu * mi;
        }
        s[b] = smax;
    }
}
