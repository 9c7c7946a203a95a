/*
 * Counter-based synthetic replay rows.
 *
 * The paper's throughput tables are measured on PyBullet/Gym locomotion tasks
 * (Section 4.1); no environment is available here, and the network update only
 * ever consumes replay rows, so the rows are drawn from the distributions the
 * workload descriptions fix:
 *   obs, next_obs ~ N(0,1)  (optionally every column j with j % zero_mod == 0 is 0)
 *   action        ~ U[-1, 1)
 *   reward        ~ N(0,1)
 *   done          ~ Bernoulli(p_done), stored as 0.0 / 1.0
 *
 * Every value is a pure function of (seed, row, field, column), so any row can be
 * regenerated without materialising the buffer. The hash is the SplitMix64 output
 * mixer (Steele, Lea, Flood, "Fast splittable pseudorandom number generators",
 * OOPSLA 2014). Normals use the Box-Muller transform in double precision (both
 * outputs of one draw fill two adjacent columns) and are rounded once to float.
 *
 * This file holds input generation only: none of the update's arithmetic.
 */
#include <math.h>
#include <stdint.h>

#define FIELD_OBS 1u
#define FIELD_ACT 2u
#define FIELD_REW 3u
#define FIELD_DONE 4u
#define FIELD_NOBS 5u

static inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

static inline uint64_t draw(uint64_t seed, uint64_t row, uint32_t field, uint32_t col) {
  uint64_t h = mix64(seed * 0x9E3779B97F4A7C15ull + 0x632BE59BD9B4E019ull);
  h = mix64(h ^ (row * 0xD1B54A32D192ED03ull));
  return mix64(h ^ (((uint64_t)field << 32) | col));
}

/* Two independent N(0,1) values from one 64-bit draw (both Box-Muller outputs). */
static inline void normal_pair(uint64_t z, float* c, float* s) {
  double u1 = ((double)(z >> 40) + 1.0) * 0x1p-24;            /* (0, 1] */
  double u2 = (double)((z >> 8) & 0xFFFFFFull) * 0x1p-24;      /* [0, 1) */
  double r = sqrt(-2.0 * log(u1)), a = 6.283185307179586 * u2;
  *c = (float)(r * cos(a));
  *s = (float)(r * sin(a));
}

static inline float uniform_pm1(uint64_t z) {
  return (float)((double)(z >> 40) * 0x1p-23 - 1.0);          /* [-1, 1) */
}

static void normals(uint64_t seed, int64_t row, uint32_t field, int32_t O, int32_t zero_mod,
                    float* out) {
  for (int32_t j = 0; j < O; j += 2) {
    float c, s;
    normal_pair(draw(seed, (uint64_t)row, field, (uint32_t)(j >> 1)), &c, &s);
    out[j] = (zero_mod > 0 && j % zero_mod == 0) ? 0.0f : c;
    if (j + 1 < O) out[j + 1] = (zero_mod > 0 && (j + 1) % zero_mod == 0) ? 0.0f : s;
  }
}

static void one_row(uint64_t seed, int64_t row, int32_t O, int32_t A, int32_t zero_mod,
                    double p_done, float* obs, float* act, float* rew, float* done,
                    float* nobs) {
  normals(seed, row, FIELD_OBS, O, zero_mod, obs);
  normals(seed, row, FIELD_NOBS, O, zero_mod, nobs);
  for (int32_t j = 0; j < A; ++j)
    act[j] = uniform_pm1(draw(seed, (uint64_t)row, FIELD_ACT, (uint32_t)j));
  float r, unused;
  normal_pair(draw(seed, (uint64_t)row, FIELD_REW, 0), &r, &unused);
  *rew = r;
  uint64_t zd = draw(seed, (uint64_t)row, FIELD_DONE, 0);
  *done = ((double)(zd >> 11) * 0x1p-53) < p_done ? 1.0f : 0.0f;
}

/* Rows row0 .. row0+n-1 into dense row-major arrays [n,O], [n,A], [n], [n], [n,O]. */
void synth_rows(uint64_t seed, int32_t O, int32_t A, int32_t zero_mod, double p_done,
                int64_t row0, int64_t n, float* obs, float* act, float* rew, float* done,
                float* nobs) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    one_row(seed, row0 + i, O, A, zero_mod, p_done, obs + i * O, act + i * A, rew + i,
            done + i, nobs + i * O);
}

/* The rows listed in rows[0..n) (any order, repeats allowed). */
void synth_rows_at(uint64_t seed, int32_t O, int32_t A, int32_t zero_mod, double p_done,
                   const int64_t* rows, int64_t n, float* obs, float* act, float* rew,
                   float* done, float* nobs) {
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i)
    one_row(seed, rows[i], O, A, zero_mod, p_done, obs + i * O, act + i * A, rew + i,
            done + i, nobs + i * O);
}
