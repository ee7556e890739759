/* Seeded synthetic workload generator for the MPCache decode/prefill path.
 *
 * This module produces the inputs (window queries, prompt K/V, decode queries) that both the CPU
 * oracle and the GPU library consume. It holds none of the method's arithmetic: it only draws
 * numbers and shapes them like the workloads the paper evaluates on (attention sinks, heavy
 * hitters, outlier key channels, rotary position embedding).
 *
 * Host and device entry points run the same __host__ __device__ element functions, so a host
 * buffer and a device buffer generated from the same spec hold the same bytes:
 *   - random bits: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC 2011), counter = element id;
 *   - normal variates: the sum of twelve uniforms minus six (Irwin-Hall, n = 12), computed exactly
 *     on 16-bit uniforms, so no transcendental function is involved;
 *   - rotary angles: a cos/sin table computed once on the host and copied to the device;
 *   - everything else: IEEE add/mul/div/sqrt in a fixed order, with FMA contraction disabled.
 *
 * Layouts are row-major and contiguous:
 *   q_win [B][Hq][W][d]  (rows = absolute positions T-W .. T-1), one layer per call on the host;
 *   k, v  [B][Hkv][T][d], one layer per call on the host;
 *   dec_q [L][B][Hq][d]  for one decode step.
 * Device entry points take whole [L][...] tensors for layers [layer0, layer0 + n_layers).
 */
#ifndef MPC_SYNTH_H
#define MPC_SYNTH_H
#include <stdint.h>
#ifdef __cplusplus
extern "C" {
#endif

enum { SYNTH_FP32 = 0, SYNTH_FP16 = 1, SYNTH_BF16 = 2 };

typedef struct {
  uint64_t seed;        /* base seed; sequence b uses seed + seq_stride * b            */
  uint64_t seq_stride;  /* 0: one key for the whole batch                              */
  int32_t n_layers, batch, n_q_heads, n_kv_heads, head_dim;
  int32_t dtype;        /* SYNTH_FP32 / SYNTH_FP16 / SYNTH_BF16                         */
  int32_t T;            /* rows of K/V (prompt length, or kept length for a direct cache) */
  int32_t W;            /* window query rows at positions T-W..T-1 (0 = none)          */
  int32_t n_outlier;    /* outlier key channels per kv head                            */
  float outlier_scale;  /* their scale (std)                                           */
  int32_t rope;         /* 1: rotate K and window Q rows by position                   */
  float rope_base;
  int32_t n_sinks;      /* positions 0..n_sinks-1 become attention sinks               */
  int32_t hh_count;     /* heavy-hitter spans                                          */
  int32_t hh_span;      /* tokens per span (1 = single tokens)                         */
  int32_t hh_lo, hh_hi; /* spans are placed in [hh_lo, hh_hi)                          */
} synth_spec;

/* Returns 0 on success, nonzero on an invalid spec / argument. */
int synth_validate(const synth_spec* sp);
int synth_rope_table(int32_t T, int32_t d, double base, double* out /* [T][d/2][2] (cos, sin) */);
int synth_outlier_channels(const synth_spec* sp, int32_t layer, int32_t b, int32_t kvh, int32_t* ch);
int synth_hh_starts(const synth_spec* sp, int32_t layer, int32_t b, int32_t kvh, int32_t* starts);

int synth_qwin_host(const synth_spec* sp, int32_t layer, const double* rope, void* out);
int synth_unit_dir_host(const synth_spec* sp, const void* qwin_layer, double* u /* [B][Hkv][d] */);
int synth_kv_host(const synth_spec* sp, int32_t layer, const void* qwin_layer, const double* rope,
                  void* k, void* v);
int synth_dq_host(const synth_spec* sp, int32_t step, void* q);

int synth_qwin_dev(const synth_spec* sp, int32_t layer0, int32_t n_layers, const double* rope_dev,
                   void* out, void* stream);
int synth_kv_dev(const synth_spec* sp, int32_t layer0, int32_t n_layers, const void* qwin_dev,
                 const double* rope_dev, double* u_ws /* [B][Hkv][d] */, void* k, void* v,
                 void* stream);
int synth_dq_dev(const synth_spec* sp, int32_t step, void* q, void* stream);

#ifdef __cplusplus
}
#endif
#endif
