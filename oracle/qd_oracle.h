/*
 * qd_oracle.h -- declarations of the CPU oracle for one MAP-Elites generation.
 *
 * TEST INFRASTRUCTURE ONLY.  This header belongs to the oracle and to nothing
 * else: the HIP library has its own header and shares no declaration, constant
 * or helper with this one.  Only the test-suite, the smoke check and the CPU
 * baseline of the benchmark load the oracle.
 */
#ifndef QD_ORACLE_H
#define QD_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Tasks and tessellations, numbered as the library numbers them (the values
 * are the interface, not shared code). */
enum { OR_RASTRIGIN = 0, OR_SPHERE = 1, OR_RASTRIGIN_PROJ = 2, OR_MLP = 3 };
enum { OR_GRID = 0, OR_CVT = 1 };

/* Rows of the Gaussian sampler's table (sixteen per binade of k = 1..2^24,
 * and one for k = 2^24). */
#define OR_NORMAL_ROWS 385

typedef struct {
  int32_t task, tess;
  int32_t n;            /* genotype length; ignored for OR_MLP (derived)       */
  int32_t batch;        /* N_B offspring per generation                         */
  int32_t D;            /* descriptor dimension, 1..4                           */
  int32_t grid[4];      /* bins per descriptor dimension (grid tessellation)    */
  int32_t C;            /* number of cells                                      */
  float lo[4], hi[4];   /* descriptor box                                       */
  float iso_sigma, line_sigma;
  float init_lo, init_hi;
  int32_t obs, hid, act, T;   /* MLP policy and rollout                         */
  int32_t cvt_samples;  /* CVT: Lloyd iterations over this many uniform points  */
  int32_t cvt_iters;    /*      (0 = centroids stay the uniform draws)          */
  int32_t death_mode;   /* policies: 0 none, 1 truncate at failure, 2 discard   */
  float death_below;    /*   failure: new state component 0 below this          */
  int32_t init_mode;    /* test functions' first batch: 0 every gene U[lo, hi);  */
                        /*   1 as 0 plus one level per genotype half, uniform   */
                        /*   over that descriptor dimension's box               */
  uint64_t seed;
} or_config;

typedef struct or_state or_state;

/* ---- primitives (exported so that the pin tests can reach each one) ---- */
void     or_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);
float    or_u24(uint32_t x);
float    or_u24p(uint32_t x);
float    or_normal(uint32_t x);               /* one standard normal per word */
double   or_normal_quantile(double p);        /* Phi^-1(1 - p/2), fp64        */
void     or_normal_table(float* out);         /* [OR_NORMAL_ROWS][4]          */
float    or_rsinpi(float x);          /* sqrt(20) sin(pi x), up to sign */
void     or_rsin_coef(float out[6]);  /* its six polynomial coefficients */
float    or_expf(float x);
float    or_tanhf(float x);
float    or_sigmoidf(float x);
float    or_r64_sum(const float* t, int32_t a, int32_t b);
void     or_eval_testfn(int32_t task, const float* x, int32_t n, const float* lo,
                        const float* hi, float* fit, float* desc);
int32_t  or_grid_cell(const float* d, int32_t D, const int32_t* grid, const float* lo,
                      const float* hi);
int32_t  or_cvt_cell(const float* d, int32_t D, const float* lo, const float* hi,
                     const float* cent, int32_t C);
void     or_mlp_rollout(const float* w, int32_t obs, int32_t hid, int32_t act, int32_t T,
                        const float* A, const float* B, const float* s0, int32_t death_mode,
                        float death_below, float* fit, float* desc);
uint64_t or_key(float f, int32_t j, int32_t batch);
void     or_map_f32(int32_t fn, const float* in, float* out, int64_t count);
void     or_philox_many(const uint32_t* ctr, const uint32_t key[2], uint32_t* out,
                        int64_t count);
void     or_normal_many(const uint32_t* x, float* out, int64_t count);

/* Threads of the per-offspring loops (OpenMP; insertion always runs in one
 * thread).  n <= 0 leaves the current setting; returns the number in use. */
int32_t   or_set_threads(int32_t n);

/* ---- the run ---- */
int32_t   or_genotype_len(const or_config* cfg);
int32_t   or_env_len(const or_config* cfg);
or_state* or_new(const or_config* cfg, int32_t keep_offspring);
void      or_free(or_state* s);
void      or_setup(or_state* s);                   /* centroids and environment   */
int32_t   or_init(or_state* s);                    /* setup + generation 0        */
int32_t   or_generation(or_state* s, uint32_t g);  /* one generation, g >= 1      */
int32_t   or_offspring(or_state* s, uint32_t g, int32_t j, float* geno, float* fit,
                       float* desc, int32_t* parents);
int32_t   or_offspring_many(or_state* s, uint32_t g, const int32_t* js, int32_t count,
                            float* fit, float* desc, int32_t* parents);
int32_t   or_insert_driven(or_state* s, const float* fit, const float* desc,
                           const float* geno, int32_t nb, int32_t* cell, uint8_t* won);
void      or_stats(const or_state* s, double offset, double out[3]);

/* views onto the state (row-major, owned by the state) */
float*   or_archive_geno(or_state* s);
float*   or_archive_fit(or_state* s);
float*   or_archive_desc(or_state* s);
uint8_t* or_archive_occ(or_state* s);
float*   or_centroids(or_state* s);
float*   or_env(or_state* s);
int32_t* or_off_parents(or_state* s);
float*   or_off_fit(or_state* s);
float*   or_off_desc(or_state* s);
int32_t* or_off_cell(or_state* s);
uint8_t* or_off_won(or_state* s);
float*   or_off_geno(or_state* s);

#ifdef __cplusplus
}
#endif
#endif
