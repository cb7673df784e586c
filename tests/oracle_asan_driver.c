/* Host sanitizer run of the oracle (oracle/gefen_oracle.c), built with address and
 * undefined-behaviour sanitizers by tests/test_oracle_sanitizers_cpu.py together with
 * the oracle's own source file. Test infrastructure only.
 *
 * Calls every oracle entry point on small seeded inputs that reach its edges: tensors
 * of 1 element, primes and highly composite sizes (Alg. 2), zero and one-element
 * blocks, blocks that are all zero (the histogram skips them, the step keeps scale 0),
 * histograms with fewer non-empty bins than entries (the degenerate DP) and a full one
 * (Alg. 3), fp32 and bf16 gradients, the quantised and unquantised step (Alg. 1) and
 * the Gefen-Muon codec. Prints "ok" when every call returned; a sanitizer report ends
 * the process with a non-zero status first. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int64_t oracle_divisors(int64_t n, int64_t* out, int64_t cap);
int oracle_partition(const void* g, int32_t dtype, int64_t n, double eps, int64_t* divs,
                     double* scores, int64_t cap, int64_t* n_div_out, int64_t* period_out);
void oracle_histogram_blocks(const void* g, int32_t dtype, const int64_t* offs,
                             int64_t nblocks, int32_t nbins, uint64_t* hist);
void oracle_histogram_uniform(const void* g, int32_t dtype, int64_t n, int64_t p,
                              int32_t nbins, uint64_t* hist);
int oracle_dp_codebook(const uint64_t* hist, int32_t nbins, int32_t k, double* codebook,
                       double* cost, int32_t* bounds);
void oracle_step_blocks(double* theta, const void* g, int32_t dtype, uint8_t* codes,
                        double* s, double* v, const int64_t* offs, int64_t nblocks,
                        const double* cb_dec, const double* cb_enc, int32_t k, double lr,
                        double beta1, double beta2, double eps, double wd, int64_t t,
                        int32_t quantize, double* m_full, double* m_out);
void oracle_step_uniform(double* theta, const void* g, int32_t dtype, uint8_t* codes,
                         double* s, double* v, int64_t n, int64_t p, const double* cb_dec,
                         const double* cb_enc, int32_t k, double lr, double beta1,
                         double beta2, double eps, double wd, int64_t t, int32_t quantize,
                         double* m_full, double* m_out);
void oracle_muon_codec_blocks(const void* g, int32_t dtype, uint8_t* codes, double* s,
                              const int64_t* offs, int64_t nblocks, const double* cb_dec,
                              const double* cb_enc, int32_t k, double mu, int32_t nesterov,
                              double* u);

static uint64_t rng_state = 0x9e3779b97f4a7c15ull;

static double unif(void)   /* xorshift64*, in (0, 1) */
{
    rng_state ^= rng_state >> 12;
    rng_state ^= rng_state << 25;
    rng_state ^= rng_state >> 27;
    return ((double)((rng_state * 0x2545f4914f6cdd1dull) >> 11) + 0.5) / 9007199254740992.0;
}

static double normal(void)
{
    return sqrt(-2.0 * log(unif())) * cos(6.283185307179586 * unif());
}

/* n gradient values (fp32 or bf16 bit patterns), every `zero_every`-th block of `blk`
 * elements all zero */
static void *grads(int64_t n, int32_t dtype, int64_t blk, int64_t zero_every)
{
    void* g = malloc((size_t)(n > 0 ? n : 1) * (dtype == 0 ? 4 : 2));
    for (int64_t i = 0; i < n; ++i) {
        int zero = blk > 0 && zero_every > 0 && (i / blk) % zero_every == 0;
        float x = zero ? 0.0f : (float)(normal() * exp(-3.0 * unif()));
        if (dtype == 0) {
            ((float*)g)[i] = x;
        } else {
            uint32_t b;
            memcpy(&b, &x, 4);
            ((uint16_t*)g)[i] = (uint16_t)((b + 0x7fffu + ((b >> 16) & 1u)) >> 16);
        }
    }
    return g;
}

static void linear_codebook(double* cb, int32_t k)
{
    for (int32_t i = 0; i < k; ++i) cb[i] = -1.0 + 2.0 * i / (k - 1);
}

static void partitions(void)
{
    static const int64_t sizes[] = {1, 2, 7, 12, 97, 360, 1024, 5040};
    int64_t divs[256], nd = 0, per = 0;
    double scores[256];
    for (size_t i = 0; i < sizeof sizes / sizeof sizes[0]; ++i)
        for (int32_t dt = 0; dt < 2; ++dt) {
            void* g = grads(sizes[i], dt, 0, 0);
            if (oracle_partition(g, dt, sizes[i], 1e-8, divs, scores, 256, &nd, &per) != 0)
                abort();
            if (oracle_partition(g, dt, sizes[i], 1e-8, divs, scores, 1, &nd, &per) == 0 &&
                nd > 1)
                abort();   /* a too small cap must be refused */
            free(g);
        }
    if (oracle_divisors(0, divs, 256) != 0 || oracle_divisors(1, divs, 0) != 1) abort();
}

static void histograms_and_dp(void)
{
    int64_t offs[] = {0, 1, 1, 33, 33, 100, 2100, 2101};   /* empty and 1-element blocks */
    const int64_t nb = 7, n = offs[nb];
    for (int32_t dt = 0; dt < 2; ++dt) {
        void* g = grads(n, dt, 0, 0);
        for (int32_t k = 2; k <= 256; k = k < 16 ? k * 2 : k * 4) {
            int32_t nbins = 16 * k;
            uint64_t* h = calloc((size_t)nbins, sizeof(uint64_t));
            oracle_histogram_blocks(g, dt, offs, nb, nbins, h);
            double* cb = malloc(sizeof(double) * (size_t)k);
            int32_t* bounds = malloc(sizeof(int32_t) * (size_t)k);
            double cost = 0.0;
            if (oracle_dp_codebook(h, nbins, k, cb, &cost, bounds) < 0) abort();
            /* degenerate: one non-empty bin, then an empty histogram */
            memset(h, 0, sizeof(uint64_t) * (size_t)nbins);
            h[nbins / 2] = 5;
            if (oracle_dp_codebook(h, nbins, k, cb, &cost, bounds) < 0) abort();
            h[nbins / 2] = 0;
            (void)oracle_dp_codebook(h, nbins, k, cb, &cost, bounds);
            free(cb);
            free(bounds);
            free(h);
        }
        uint64_t hu[64] = {0};
        oracle_histogram_uniform(g, dt, 2100, 21, 64, hu);
        free(g);
    }
    uint64_t h1[4] = {1, 0, 0, 3};
    double cb[2];
    int32_t bd[2];
    double cost;
    if (oracle_dp_codebook(h1, 4, 1, cb, &cost, bd) != -1) abort();   /* k < 2 refused */
    (void)oracle_dp_codebook(h1, 4, 2, cb, &cost, bd);
}

static void steps(void)
{
    int64_t offs[] = {0, 1, 3, 35, 35, 300, 301, 1301};
    const int64_t nb = 7, n = offs[nb];
    const int32_t k = 256;
    double cb[256];
    linear_codebook(cb, k);
    for (int32_t dt = 0; dt < 2; ++dt)
        for (int32_t quant = 0; quant < 2; ++quant) {
            void* g = grads(n, dt, 35, 2);   /* some all-zero blocks */
            double* th = calloc((size_t)n, sizeof(double));
            double* m_full = calloc((size_t)n, sizeof(double));
            double* m_out = calloc((size_t)n, sizeof(double));
            uint8_t* codes = calloc((size_t)n, 1);
            double s[7] = {0}, v[7] = {0};
            for (int64_t t = 1; t <= 3; ++t)
                oracle_step_blocks(th, g, dt, codes, s, v, offs, nb, cb, cb, k, 1e-3, 0.9,
                                   0.999, 1e-8, 0.1, t, quant, m_full, m_out);
            double su[8] = {0}, vu[8] = {0};
            oracle_step_uniform(th, g, dt, codes, su, vu, 1296, 162, cb, cb, k, 1e-3, 0.9,
                                0.999, 1e-8, 0.1, 4, quant, m_full, m_out);
            double* u = calloc((size_t)n, sizeof(double));
            oracle_muon_codec_blocks(g, dt, codes, s, offs, nb, cb, cb, k, 0.95, dt, u);
            free(u);
            free(g);
            free(th);
            free(m_full);
            free(m_out);
            free(codes);
        }
}

int main(void)
{
    partitions();
    histograms_and_dp();
    steps();
    puts("ok");
    return 0;
}
