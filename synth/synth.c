/*
 * synth.c -- seeded synthetic replica gradients for the detect-and-aggregate
 * step.  This is the ONE input generator: both the oracle and the HIP path
 * consume the bytes it writes.  It holds none of the method's arithmetic
 * (no comparison, vote, clique, selection or reduction): it only turns a
 * per-replica role table into numbers.
 *
 * Random numbers: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random
 * numbers: as easy as 1, 2, 3", SC'11), counter-based, so any coordinate
 * range can be generated independently and in any order.
 *
 * Values (the workload shapes of the paper's CIFAR-10 / ResNet-18 runs):
 *   honest   g_i[k] = fl32(0.01 * Z)  with Z ~ N(0,1)        (dist 0)
 *                     fl32(0.01 * T)  with T ~ Student-t(3)  (dist 1)
 *   reversed -100 * g_i[k]                       (reversed-gradient attack)
 *   ALIE     fl32(mu_k - z * sigma_k), mu/sigma = mean and population std
 *            of the f honest g_i[k] in fp64, ascending i (same vector for
 *            every colluder and file)
 *   noise    fl32(N(0,1)), independent per (worker, file, coordinate)
 * All honest replicas of a file are copies of the same bits.
 */
#include "synth.h"

#include <math.h>
#include <pthread.h>
#include <stdlib.h>
#include <string.h>

/* ---- Philox4x32-10 ------------------------------------------------- */
#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

static void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2],
                          uint32_t out[4])
{
    uint32_t c0 = ctr_in[0], c1 = ctr_in[1], c2 = ctr_in[2], c3 = ctr_in[3];
    uint32_t k0 = key_in[0], k1 = key_in[1];
    for (int round = 0; round < 10; ++round) {
        uint64_t p0 = (uint64_t)PHILOX_M0 * c0;
        uint64_t p1 = (uint64_t)PHILOX_M1 * c2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        uint32_t n0 = hi1 ^ c1 ^ k0;
        uint32_t n1 = lo1;
        uint32_t n2 = hi0 ^ c3 ^ k1;
        uint32_t n3 = lo0;
        c0 = n0; c1 = n1; c2 = n2; c3 = n3;
        k0 += PHILOX_W0;
        k1 += PHILOX_W1;
    }
    out[0] = c0; out[1] = c1; out[2] = c2; out[3] = c3;
}

void synth_philox(uint64_t seed, const uint32_t ctr[4], uint32_t out[4])
{
    uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
    philox4x32_10(ctr, key, out);
}

/* uniform in (0,1) from 64 random bits, 53-bit resolution */
static double unit_open(uint32_t hi, uint32_t lo)
{
    uint64_t v = (((uint64_t)hi << 32) | lo) >> 11;
    return ((double)v + 0.5) * (1.0 / 9007199254740992.0);
}

/* Two standard normals by Box-Muller from one Philox block. */
static void normal_pair(uint64_t seed, uint32_t a, uint32_t b, uint32_t c,
                        uint32_t d, double z[2])
{
    uint32_t ctr[4] = { a, b, c, d }, x[4];
    synth_philox(seed, ctr, x);
    double u1 = unit_open(x[0], x[1]);
    double u2 = unit_open(x[2], x[3]);
    double rad = sqrt(-2.0 * log(u1));
    double ang = 6.283185307179586476925286766559 * u2;
    z[0] = rad * cos(ang);
    z[1] = rad * sin(ang);
}

/* Standard normal for (stream, file, coordinate). */
static double normal_at(uint64_t seed, uint32_t stream, uint32_t file,
                        uint64_t k)
{
    double z[2];
    uint64_t pair = k >> 1;
    normal_pair(seed, (uint32_t)pair, (uint32_t)(pair >> 32), file,
                stream << 4, z);
    return z[k & 1];
}

/* Student-t with 3 degrees of freedom: Z0 / sqrt((Z1^2+Z2^2+Z3^2)/3). */
static double student3_at(uint64_t seed, uint32_t stream, uint32_t file,
                          uint64_t k)
{
    double za[2], zb[2];
    normal_pair(seed, (uint32_t)k, (uint32_t)(k >> 32), file,
                (stream << 4) | 1u, za);
    normal_pair(seed, (uint32_t)k, (uint32_t)(k >> 32), file,
                (stream << 4) | 2u, zb);
    double chi = za[1] * za[1] + zb[0] * zb[0] + zb[1] * zb[1];
    return za[0] / sqrt(chi / 3.0);
}

float synth_honest_value(uint64_t seed, int32_t dist, uint32_t file, uint64_t k)
{
    double v = dist == SYNTH_DIST_STUDENT3 ? student3_at(seed, 1u, file, k)
                                           : normal_at(seed, 1u, file, k);
    return (float)(0.01 * v);
}

float synth_noise_value(uint64_t seed, uint32_t worker, uint32_t file, uint64_t k)
{
    return (float)normal_at(seed, 2u + worker, file, k);
}

uint32_t synth_u32(uint64_t seed, uint32_t stream, uint64_t index)
{
    uint32_t ctr[4] = { (uint32_t)index, (uint32_t)(index >> 32), 0xA5A5A5A5u,
                        stream }, x[4];
    synth_philox(seed, ctr, x);
    return x[0];
}

/* ---- chunk fill ---------------------------------------------------- */

typedef struct {
    const uint8_t *role;
    const int32_t *worker;
    int64_t f;
    int32_t r;
    int64_t k0, nk;      /* chunk coordinates [k0, k0+nk)              */
    int64_t j0, j1;      /* this thread's sub-range of [0, nk)         */
    int32_t dist;
    uint64_t seed;
    double alie_z;
    float *out;          /* [f][r][nk]                                 */
    float *honest;       /* scratch [f][nk]                            */
    int need_alie;
} fill_job;

static void *fill_worker(void *arg)
{
    fill_job *J = (fill_job *)arg;
    const int64_t f = J->f, nk = J->nk;
    const int32_t r = J->r;
    for (int64_t i = 0; i < f; ++i)
        for (int64_t j = J->j0; j < J->j1; ++j)
            J->honest[i * nk + j] =
                synth_honest_value(J->seed, J->dist, (uint32_t)i, (uint64_t)(J->k0 + j));

    float *alie = NULL;
    if (J->need_alie) {
        alie = (float *)malloc((size_t)(J->j1 - J->j0) * sizeof(float));
        for (int64_t j = J->j0; j < J->j1; ++j) {
            double mu = 0.0, var = 0.0;
            for (int64_t i = 0; i < f; ++i) mu += (double)J->honest[i * nk + j];
            mu /= (double)f;
            for (int64_t i = 0; i < f; ++i) {
                double dv = (double)J->honest[i * nk + j] - mu;
                var += dv * dv;
            }
            double sigma = sqrt(var / (double)f);
            alie[j - J->j0] = (float)(mu - J->alie_z * sigma);
        }
    }

    for (int64_t i = 0; i < f; ++i)
        for (int32_t s = 0; s < r; ++s) {
            float *row = J->out + (i * r + s) * nk;
            const float *hv = J->honest + i * nk;
            uint8_t role = J->role[i * r + s];
            int32_t w = J->worker[i * r + s];
            for (int64_t j = J->j0; j < J->j1; ++j) {
                float v;
                switch (role) {
                case SYNTH_ROLE_REVERSED: v = -100.0f * hv[j]; break;
                case SYNTH_ROLE_ALIE:     v = alie[j - J->j0]; break;
                case SYNTH_ROLE_NOISE:
                    v = synth_noise_value(J->seed, (uint32_t)w, (uint32_t)i,
                                          (uint64_t)(J->k0 + j));
                    break;
                default:                  v = hv[j]; break;
                }
                row[j] = v;
            }
        }
    free(alie);
    return NULL;
}

int synth_fill(const uint8_t *role, const int32_t *worker, int64_t f, int32_t r,
               int64_t k0, int64_t nk, int32_t dist, uint64_t seed,
               double alie_z, float *out, int32_t nthreads)
{
    if (!role || !worker || !out || f <= 0 || r <= 0 || k0 < 0 || nk < 0)
        return -1;
    if (nk == 0) return 0;
    if (nthreads < 1) nthreads = 1;
    if (nthreads > 256) nthreads = 256;
    if (nthreads > nk) nthreads = (int32_t)nk;
    int need_alie = 0;
    for (int64_t x = 0; x < f * r; ++x) need_alie |= role[x] == SYNTH_ROLE_ALIE;
    float *honest = (float *)malloc((size_t)(f * nk) * sizeof(float));
    if (!honest) return -2;
    fill_job jobs[256];
    pthread_t tids[256];
    for (int32_t t = 0; t < nthreads; ++t) {
        fill_job *J = &jobs[t];
        J->role = role; J->worker = worker; J->f = f; J->r = r;
        J->k0 = k0; J->nk = nk;
        J->j0 = nk * t / nthreads; J->j1 = nk * (t + 1) / nthreads;
        J->dist = dist; J->seed = seed; J->alie_z = alie_z;
        J->out = out; J->honest = honest; J->need_alie = need_alie;
    }
    for (int32_t t = 1; t < nthreads; ++t)
        pthread_create(&tids[t], NULL, fill_worker, &jobs[t]);
    fill_worker(&jobs[0]);
    for (int32_t t = 1; t < nthreads; ++t) pthread_join(tids[t], NULL);
    free(honest);
    return 0;
}

/* FNV-1a over the bytes of a float buffer: logged by tests so both sides
 * demonstrably consumed the same input. */
uint64_t synth_fnv1a(const void *buf, int64_t nbytes)
{
    const uint8_t *p = (const uint8_t *)buf;
    uint64_t h = 1469598103934665603ull;
    for (int64_t i = 0; i < nbytes; ++i) {
        h ^= p[i];
        h *= 1099511628211ull;
    }
    return h;
}
