/*
 * synth.hip -- seeded synthetic replica gradients for the detect-and-
 * aggregate step.  This is the ONE input generator: both the oracle and the
 * HIP path consume what it writes.  It holds none of the method's arithmetic
 * (no comparison, vote, clique, selection or reduction): it only turns a
 * per-replica role table into numbers.
 *
 * The same value functions run on the host (pthreads) and on the GPU, and
 * give the same bits on both: they use integer operations and IEEE-754
 * double add / multiply / divide / square root only (all correctly rounded),
 * and this file is compiled with floating-point contraction off.
 *
 * Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), counter-based, so any coordinate
 * range can be generated independently, in any order, on either side.
 *
 * Standard normal deviates: the polar method (Marsaglia and Bray, "A
 * convenient method for generating normal variables", SIAM Review 6, 1964):
 * a point (v1, v2) uniform in the square [-1, 1)^2 from one Philox block,
 * again from the next block while s = v1^2 + v2^2 is outside (0, 1), then
 * Z = v1 * sqrt(-2 ln(s) / s).  The logarithm is computed here from the
 * double's exponent and the series 2 atanh(t) of its mantissa (basic
 * operations only, so both sides round alike).
 *
 * Values (the workload shapes of the paper's CIFAR-10 / ResNet-18 runs):
 *   honest   g_i[k] = fl32(0.01 * Z)                         (dist 0)
 *                     fl32(0.01 * Z0 / sqrt((Z1^2+Z2^2+Z3^2)/3)), a
 *                     Student-t with 3 degrees of freedom     (dist 1)
 *                     the binary32 pattern 0x3F800000 | (16 random bits),
 *                     values in [1, 1 + 2^-7) sharing their high 16 bits
 *                                                             (dist 2)
 *   reversed -100 * g_i[k] (binary32 multiply)
 *   ALIE     fl32(mu_k - z * sigma_k): mean and population std of the f
 *            honest g_i[k], fp64, files in ascending order (same vector for
 *            every colluder and file)
 *   noise    fl32(Z), independent per (worker, file, coordinate)
 * All honest replicas of a file are copies of the same bits.
 */
#include <hip/hip_runtime.h>
#include <pthread.h>

#include <cstdint>
#include <cstdlib>
#include <cstring>

#include "synth.h"

namespace {

constexpr uint32_t kM0 = 0xD2511F53u, kM1 = 0xCD9E8D57u;
constexpr uint32_t kW0 = 0x9E3779B9u, kW1 = 0xBB67AE85u;

struct U4 {
    uint32_t x[4];
};

__host__ __device__ inline U4 philox(uint64_t seed, uint32_t c0, uint32_t c1, uint32_t c2,
                                     uint32_t c3) {
    uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    for (int round = 0; round < 10; ++round) {
        const uint64_t p0 = (uint64_t)kM0 * c0;
        const uint64_t p1 = (uint64_t)kM1 * c2;
        const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c1 ^ k0;
        const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c3 ^ k1;
        c1 = (uint32_t)p1;
        c3 = (uint32_t)p0;
        c0 = n0;
        c2 = n2;
        k0 += kW0;
        k1 += kW1;
    }
    return U4{{c0, c1, c2, c3}};
}

// Natural logarithm of a positive normal double, from x = m * 2^e with m in
// [sqrt(1/2), sqrt(2)]: ln x = e ln 2 + 2 atanh(t), t = (m - 1) / (m + 1),
// |t| <= 0.1716, the series to t^25 (the next term is below 1e-20 of it).
__host__ __device__ inline double log_pos(double x) {
    uint64_t b;
    __builtin_memcpy(&b, &x, sizeof b);
    int e = (int)((b >> 52) & 0x7FFu) - 1023;
    b = (b & 0x000FFFFFFFFFFFFFull) | 0x3FF0000000000000ull;
    double m;
    __builtin_memcpy(&m, &b, sizeof m);
    if (m > 1.4142135623730951) {
        m *= 0.5;
        ++e;
    }
    const double t = (m - 1.0) / (m + 1.0);
    const double t2 = t * t;
    double p = 1.0 / 25.0;
    for (int j = 11; j >= 0; --j) p = p * t2 + 1.0 / (double)(2 * j + 1);
    return (double)e * 0.69314718055994530942 + 2.0 * t * p;
}

// A double in [0, 1) from 53 random bits of two words (exact).
__host__ __device__ inline double uniform53(uint32_t a, uint32_t b) {
    return ((double)(a >> 5) * 67108864.0 + (double)(b >> 6)) * (1.0 / 9007199254740992.0);
}

// Standard normal for counter (stream, sub, file, k), by the polar method:
// attempt a reads Philox block (k, file, 2^31 | stream << 16 | sub << 8 | a)
// (attempts past 255, probability below 1e-170, give 0).
__host__ __device__ inline double normal(uint64_t seed, uint32_t stream, uint32_t sub,
                                         uint32_t file, uint64_t k) {
    for (uint32_t a = 0; a < 256u; ++a) {
        const U4 u = philox(seed, (uint32_t)k, (uint32_t)(k >> 32), file,
                            0x80000000u | (stream << 16) | (sub << 8) | a);
        const double v1 = 2.0 * uniform53(u.x[0], u.x[1]) - 1.0;
        const double v2 = 2.0 * uniform53(u.x[2], u.x[3]) - 1.0;
        const double s = v1 * v1 + v2 * v2;
        if (s > 0.0 && s < 1.0) return v1 * sqrt(-2.0 * log_pos(s) / s);
    }
    return 0.0;
}

__host__ __device__ inline float honest_value(uint64_t seed, int32_t dist, uint32_t file,
                                              uint64_t k) {
    if (dist == SYNTH_DIST_TIED) {
        // 1 + (16 random bits) * 2^-23: the bit pattern 0x3F80xxxx
        const U4 u = philox(seed, (uint32_t)k, (uint32_t)(k >> 32), file, 1u << 8);
        const uint32_t bits = 0x3F800000u | (u.x[0] & 0xFFFFu);
        float v;
        __builtin_memcpy(&v, &bits, sizeof v);
        return v;
    }
    if (dist == SYNTH_DIST_STUDENT3) {
        const double z0 = normal(seed, 1u, 0u, file, k);
        const double z1 = normal(seed, 1u, 1u, file, k);
        const double z2 = normal(seed, 1u, 2u, file, k);
        const double z3 = normal(seed, 1u, 3u, file, k);
        const double chi = z1 * z1 + z2 * z2 + z3 * z3;
        return (float)(0.01 * (z0 / sqrt(chi / 3.0)));
    }
    return (float)(0.01 * normal(seed, 1u, 0u, file, k));
}

__host__ __device__ inline float noise_value(uint64_t seed, uint32_t worker, uint32_t file,
                                             uint64_t k) {
    return (float)normal(seed, 2u + worker, 0u, file, k);
}

// ALIE value of coordinate k: statistics of the f honest file gradients.
__host__ __device__ inline float alie_value(uint64_t seed, int32_t dist, int64_t f, uint64_t k,
                                            double z) {
    double mu = 0.0;
    for (int64_t i = 0; i < f; ++i) mu += (double)honest_value(seed, dist, (uint32_t)i, k);
    mu /= (double)f;
    double var = 0.0;
    for (int64_t i = 0; i < f; ++i) {
        const double dv = (double)honest_value(seed, dist, (uint32_t)i, k) - mu;
        var += dv * dv;
    }
    const double sigma = sqrt(var / (double)f);
    const double zs = z * sigma;
    return (float)(mu - zs);
}

__host__ __device__ inline float replica_value(uint8_t role, uint32_t worker, uint64_t seed,
                                               int32_t dist, uint32_t file, uint64_t k,
                                               float honest, float alie) {
    switch (role) {
    case SYNTH_ROLE_REVERSED: return -100.0f * honest;
    case SYNTH_ROLE_ALIE: return alie;
    case SYNTH_ROLE_NOISE: return noise_value(seed, worker, file, k);
    default: return honest;
    }
}

// ---------------------------------------------------------------- host fill

struct FillJob {
    const uint8_t *role;
    const int32_t *worker;
    int64_t f;
    int32_t r;
    int64_t k0, nk, j0, j1;
    int32_t dist;
    uint64_t seed;
    double alie_z;
    int need_alie;
    float *out;
};

constexpr int64_t kHostBlock = 512;   // coordinates per host work block

void *fill_worker(void *arg) {
    FillJob *J = static_cast<FillJob *>(arg);
    const int64_t f = J->f, nk = J->nk;
    float *honest = (float *)malloc((size_t)(f * kHostBlock) * sizeof(float));
    double *mu = (double *)malloc(kHostBlock * sizeof(double));
    double *var = (double *)malloc(kHostBlock * sizeof(double));
    float *alie = (float *)malloc(kHostBlock * sizeof(float));
    for (int64_t b0 = J->j0; b0 < J->j1; b0 += kHostBlock) {
        const int64_t w = (J->j1 - b0) < kHostBlock ? (J->j1 - b0) : kHostBlock;
        for (int64_t i = 0; i < f; ++i)
            for (int64_t j = 0; j < w; ++j)
                honest[i * kHostBlock + j] =
                    honest_value(J->seed, J->dist, (uint32_t)i, (uint64_t)(J->k0 + b0 + j));
        if (J->need_alie) {
            // same arithmetic as alie_value(), reusing the honest values above
            for (int64_t j = 0; j < w; ++j) mu[j] = 0.0, var[j] = 0.0;
            for (int64_t i = 0; i < f; ++i)
                for (int64_t j = 0; j < w; ++j) mu[j] += (double)honest[i * kHostBlock + j];
            for (int64_t j = 0; j < w; ++j) mu[j] /= (double)f;
            for (int64_t i = 0; i < f; ++i)
                for (int64_t j = 0; j < w; ++j) {
                    const double dv = (double)honest[i * kHostBlock + j] - mu[j];
                    var[j] += dv * dv;
                }
            for (int64_t j = 0; j < w; ++j) {
                const double sigma = sqrt(var[j] / (double)f);
                const double zs = J->alie_z * sigma;
                alie[j] = (float)(mu[j] - zs);
            }
        }
        for (int64_t i = 0; i < f; ++i)
            for (int32_t s = 0; s < J->r; ++s) {
                float *row = J->out + (i * J->r + s) * nk + b0;
                const float *hv = honest + i * kHostBlock;
                const uint8_t role = J->role[i * J->r + s];
                const uint32_t wk = (uint32_t)J->worker[i * J->r + s];
                if (role == SYNTH_ROLE_HONEST) {
                    memcpy(row, hv, (size_t)w * sizeof(float));
                    continue;
                }
                for (int64_t j = 0; j < w; ++j)
                    row[j] = replica_value(role, wk, J->seed, J->dist, (uint32_t)i,
                                           (uint64_t)(J->k0 + b0 + j), hv[j],
                                           J->need_alie ? alie[j] : 0.0f);
            }
    }
    free(honest);
    free(mu);
    free(var);
    free(alie);
    return nullptr;
}

// -------------------------------------------------------------- device fill

__global__ void alie_kernel(uint64_t seed, int32_t dist, int64_t f, int64_t d, double z,
                            float *alie) {
    for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < d;
         k += (int64_t)gridDim.x * blockDim.x)
        alie[k] = alie_value(seed, dist, f, (uint64_t)k, z);
}

__global__ void fill_kernel(const uint8_t *role, const int32_t *worker, int64_t f, int32_t r,
                            int64_t d, int32_t dist, uint64_t seed, const float *alie,
                            float *out) {
    for (int64_t i = blockIdx.y; i < f; i += gridDim.y) {
        for (int64_t k = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; k < d;
             k += (int64_t)gridDim.x * blockDim.x) {
            const float h = honest_value(seed, dist, (uint32_t)i, (uint64_t)k);
            const float a = alie ? alie[k] : 0.0f;
            for (int32_t s = 0; s < r; ++s) {
                const uint8_t ro = role[i * r + s];
                out[(i * r + s) * d + k] =
                    replica_value(ro, (uint32_t)worker[i * r + s], seed, dist, (uint32_t)i,
                                  (uint64_t)k, h, a);
            }
        }
    }
}

}  // namespace

extern "C" {

uint32_t synth_u32(uint64_t seed, uint32_t stream, uint64_t index) {
    return philox(seed, (uint32_t)index, (uint32_t)(index >> 32), 0xA5A5A5A5u, stream).x[0];
}

float synth_honest_value(uint64_t seed, int32_t dist, uint32_t file, uint64_t k) {
    return honest_value(seed, dist, file, k);
}

float synth_noise_value(uint64_t seed, uint32_t worker, uint32_t file, uint64_t k) {
    return noise_value(seed, worker, file, k);
}

double synth_normal(uint64_t seed, uint32_t stream, uint32_t sub, uint32_t file, uint64_t k) {
    return normal(seed, stream, sub, file, k);
}

double synth_log(double x) { return log_pos(x); }

int synth_fill(const uint8_t *role, const int32_t *worker, int64_t f, int32_t r, int64_t k0,
               int64_t nk, int32_t dist, uint64_t seed, double alie_z, float *out,
               int32_t nthreads) {
    if (!role || !worker || !out || f <= 0 || r <= 0 || k0 < 0 || nk < 0) return -1;
    if (nk == 0) return 0;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    if (nthreads > nk) nthreads = (int32_t)nk;
    int need_alie = 0;
    for (int64_t x = 0; x < f * r; ++x) need_alie |= role[x] == SYNTH_ROLE_ALIE;
    FillJob jobs[256];
    pthread_t tids[256];
    for (int32_t t = 0; t < nthreads; ++t) {
        jobs[t] = FillJob{role, worker, f, r, k0, nk, nk * t / nthreads, nk * (t + 1) / nthreads,
                          dist, seed, alie_z, need_alie, out};
    }
    for (int32_t t = 1; t < nthreads; ++t) pthread_create(&tids[t], nullptr, fill_worker, &jobs[t]);
    fill_worker(&jobs[0]);
    for (int32_t t = 1; t < nthreads; ++t) pthread_join(tids[t], nullptr);
    return 0;
}

int synth_fill_device(const uint8_t *role_dev, const int32_t *worker_dev, int64_t f, int32_t r,
                      int64_t d, int32_t dist, uint64_t seed, double alie_z, int32_t need_alie,
                      float *alie_dev, float *out_dev, void *stream) {
    if (!role_dev || !worker_dev || !out_dev || f <= 0 || r <= 0 || d <= 0) return -1;
    if (need_alie && !alie_dev) return -1;
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (need_alie) {
        alie_kernel<<<4096, 256, 0, s>>>(seed, dist, f, d, alie_z, alie_dev);
        if (hipGetLastError() != hipSuccess) return -3;
    }
    const int64_t bx = (d + 255) / 256;
    dim3 grid((unsigned)(bx < 1024 ? bx : 1024), (unsigned)(f < 65535 ? f : 65535));
    fill_kernel<<<grid, 256, 0, s>>>(role_dev, worker_dev, f, r, d, dist, seed,
                                     need_alie ? alie_dev : nullptr, out_dev);
    return hipGetLastError() == hipSuccess ? 0 : -3;
}

uint64_t synth_fnv1a(const void *buf, int64_t nbytes) {
    const uint8_t *p = static_cast<const uint8_t *>(buf);
    uint64_t h = 1469598103934665603ull;
    for (int64_t i = 0; i < nbytes; ++i) {
        h ^= p[i];
        h *= 1099511628211ull;
    }
    return h;
}

}  // extern "C"
