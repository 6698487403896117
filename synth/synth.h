/*
 * synth.h -- seeded synthetic replica gradients (the one input generator
 * both the oracle and the HIP path consume).  Host fill and a bit-identical
 * device fill.
 */
#ifndef ASPIS_SYNTH_H
#define ASPIS_SYNTH_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { SYNTH_ROLE_HONEST = 0, SYNTH_ROLE_REVERSED = 1, SYNTH_ROLE_ALIE = 2,
       SYNTH_ROLE_NOISE = 3 };
/* NORMAL: 0.01 * N(0,1); STUDENT3: 0.01 * t(3); TIED: 1 + u * 2^-23 with a
 * 16-bit uniform u, i.e. every value shares the high 16 bits 0x3F80 of its
 * binary32 pattern (the heaviest ties a half-key tile can meet). */
enum { SYNTH_DIST_NORMAL = 0, SYNTH_DIST_STUDENT3 = 1, SYNTH_DIST_TIED = 2 };

/* One 32-bit draw, for seeded choices (adversary sets, permutations). */
uint32_t synth_u32(uint64_t seed, uint32_t stream, uint64_t index);

/* Honest gradient g_file[k] and a noise value for (worker, file, k). */
float synth_honest_value(uint64_t seed, int32_t dist, uint32_t file, uint64_t k);
float synth_noise_value(uint64_t seed, uint32_t worker, uint32_t file, uint64_t k);
/* The standard normal deviate of a counter (polar method), and the natural
 * logarithm of a positive normal double it uses (exposed for tests). */
double synth_normal(uint64_t seed, uint32_t stream, uint32_t sub, uint32_t file, uint64_t k);
double synth_log(double x);

/* Fill out[f][r][nk] with coordinates [k0, k0+nk) of every replica.
 * role[i*r+s] picks the value of slot s of file i; worker[i*r+s] is the
 * worker holding it (only the noise role uses it).  Returns 0 on success. */
int synth_fill(const uint8_t *role, const int32_t *worker, int64_t f, int32_t r,
               int64_t k0, int64_t nk, int32_t dist, uint64_t seed,
               double alie_z, float *out, int32_t nthreads);

/* Same bytes as synth_fill for all d coordinates, written on the GPU into
 * out_dev[f][r][d].  role_dev / worker_dev are device copies of the tables;
 * alie_dev is device scratch of d floats (needed when need_alie). */
int synth_fill_device(const uint8_t *role_dev, const int32_t *worker_dev, int64_t f,
                      int32_t r, int64_t d, int32_t dist, uint64_t seed, double alie_z,
                      int32_t need_alie, float *alie_dev, float *out_dev, void *stream);

uint64_t synth_fnv1a(const void *buf, int64_t nbytes);

#ifdef __cplusplus
}
#endif
#endif
