// Seeded synthetic workload generator: host and device entry points over shared element
// functions. Built with FMA contraction off so host and device agree bit for bit.
#include "synth.h"

#include <hip/hip_runtime.h>
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define SY_HD __host__ __device__ inline

namespace {

enum : uint32_t { K_QWIN = 1, K_KEY = 2, K_VAL = 3, K_DECQ = 4, K_OUTL = 5, K_HHPOS = 6, K_HHNOISE = 7 };

// Philox4x32-10, as published by Salmon et al. (SC 2011): ten rounds of two 32x32->64-bit
// multiplies with the Weyl key schedule.
SY_HD void philox10(uint32_t c[4], uint32_t k0, uint32_t k1) {
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    const uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k0;
    const uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k1;
    c[1] = (uint32_t)p1;
    c[3] = (uint32_t)p0;
    c[0] = n0;
    c[2] = n2;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
}

struct Key {
  uint32_t k0, k1;
};

SY_HD Key seq_key(uint64_t seed, uint64_t stride, int b) {
  const uint64_t s = seed + stride * (uint64_t)b;
  return Key{(uint32_t)s, (uint32_t)(s >> 32)};
}

SY_HD uint32_t stream_id(int layer, int b, int head) {
  return (uint32_t)head | ((uint32_t)layer << 10) | ((uint32_t)b << 20);
}

// Approximately N(0,1): twelve 16-bit uniforms summed exactly, minus their mean, over 2^16.
SY_HD double normal12(Key k, uint32_t c0, uint32_t c1, uint32_t kind) {
  uint32_t a[4] = {c0, c1, kind, 0u};
  uint32_t b[4] = {c0, c1, kind, 1u};
  philox10(a, k.k0, k.k1);
  philox10(b, k.k0, k.k1);
  int64_t s = 0;
  for (int i = 0; i < 4; ++i) s += (int64_t)(a[i] & 0xFFFFu) + (int64_t)(a[i] >> 16);
  for (int i = 0; i < 2; ++i) s += (int64_t)(b[i] & 0xFFFFu) + (int64_t)(b[i] >> 16);
  return (double)(s - 393210) * (1.0 / 65536.0);
}

SY_HD uint32_t draw_u32(Key k, uint32_t c0, uint32_t c1, uint32_t kind) {
  uint32_t a[4] = {c0, c1, kind, 2u};
  philox10(a, k.k0, k.k1);
  return a[0];
}

SY_HD uint32_t f32_bits(float f) { return __builtin_bit_cast(uint32_t, f); }

SY_HD uint16_t to_bf16(float f) {
  uint32_t u = f32_bits(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

SY_HD uint16_t to_f16(float f) {
  const uint32_t x = f32_bits(f);
  const uint32_t sign = (x >> 16) & 0x8000u;
  const uint32_t ax = x & 0x7FFFFFFFu;
  if (ax > 0x7F800000u) return (uint16_t)(sign | 0x7E00u);
  if (ax >= 0x477FF000u) return (uint16_t)(sign | 0x7C00u);  // rounds to infinity
  const int e = (int)(ax >> 23);
  const uint32_t m = (ax & 0x7FFFFFu) | 0x800000u;
  if (e < 113) {  // half-precision subnormal (or zero)
    const int shift = 126 - e;
    if (shift >= 25 || ax == 0) return (uint16_t)sign;
    uint32_t q = m >> shift;
    const uint32_t rem = m & ((1u << shift) - 1u), half = 1u << (shift - 1);
    if (rem > half || (rem == half && (q & 1u))) ++q;
    return (uint16_t)(sign | q);
  }
  uint32_t h = sign | ((uint32_t)(e - 112) << 10) | ((m & 0x7FFFFFu) >> 13);
  const uint32_t rem = m & 0x1FFFu;
  if (rem > 0x1000u || (rem == 0x1000u && (h & 1u))) ++h;
  return (uint16_t)h;
}

SY_HD void store_elt(void* base, size_t idx, int dtype, double x) {
  const float f = (float)x;
  if (dtype == SYNTH_FP32)
    ((float*)base)[idx] = f;
  else if (dtype == SYNTH_BF16)
    ((uint16_t*)base)[idx] = to_bf16(f);
  else
    ((uint16_t*)base)[idx] = to_f16(f);
}

SY_HD double load_elt(const void* base, size_t idx, int dtype) {
  if (dtype == SYNTH_FP32) return (double)((const float*)base)[idx];
  const uint16_t h = ((const uint16_t*)base)[idx];
  if (dtype == SYNTH_BF16) return (double)__builtin_bit_cast(float, (uint32_t)h << 16);
  // binary16 -> double, exact
  const int e = (h >> 10) & 0x1F;
  const int mant = h & 0x3FF;
  double v;
  if (e == 0)
    v = ldexp((double)mant, -24);
  else if (e == 31)
    v = mant ? (double)NAN : (double)INFINITY;
  else
    v = ldexp((double)(mant | 0x400), e - 25);
  return (h & 0x8000) ? -v : v;
}

SY_HD void rotate(double* x, double* y, const double* cs) {
  const double a = *x * cs[0];
  const double b = *y * cs[1];
  const double c = *x * cs[1];
  const double d = *y * cs[0];
  *x = a - b;
  *y = c + d;
}

// Row of window queries at absolute position p for q-head h. Writes d values to `out`.
SY_HD void qwin_row(const synth_spec& sp, int layer, int b, int h, int p, const double* rope,
                    void* out, size_t off) {
  const Key key = seq_key(sp.seed, sp.seq_stride, b);
  const uint32_t sid = stream_id(layer, b, h);
  const int d = sp.head_dim;
  for (int i = 0; i < d; i += 2) {
    double x = normal12(key, (uint32_t)(p * d + i), sid, K_QWIN);
    double y = normal12(key, (uint32_t)(p * d + i + 1), sid, K_QWIN);
    if (sp.rope) rotate(&x, &y, rope + ((size_t)p * (d / 2) + i / 2) * 2);
    store_elt(out, off + i, sp.dtype, x);
    store_elt(out, off + i + 1, sp.dtype, y);
  }
}

SY_HD bool is_outlier(const int32_t* ch, int n, int c) {
  for (int j = 0; j < n; ++j)
    if (ch[j] == c) return true;
  return false;
}

// Key pair (c, c+1) of an unplanted row, before rounding.
SY_HD void key_pair(const synth_spec& sp, Key key, uint32_t sid, int p, int c, const int32_t* outl,
                    const double* rope, double* x, double* y) {
  const int d = sp.head_dim;
  *x = normal12(key, (uint32_t)(p * d + c), sid, K_KEY);
  *y = normal12(key, (uint32_t)(p * d + c + 1), sid, K_KEY);
  if (is_outlier(outl, sp.n_outlier, c)) *x = *x * (double)sp.outlier_scale;
  if (is_outlier(outl, sp.n_outlier, c + 1)) *y = *y * (double)sp.outlier_scale;
  if (sp.rope) rotate(x, y, rope + ((size_t)p * (d / 2) + c / 2) * 2);
}

// Planted row (sink or heavy hitter) at position p. `u` is the unit query-mean direction.
SY_HD void planted_row(const synth_spec& sp, Key key, uint32_t sid, int p, bool sink,
                       const int32_t* outl, const double* rope, const double* u, double a_sink,
                       double a_hh, double* row) {
  const int d = sp.head_dim;
  if (sink) {
    for (int c = 0; c < d; c += 2) key_pair(sp, key, sid, p, c, outl, rope, &row[c], &row[c + 1]);
    double proj = 0.0;
    for (int c = 0; c < d; ++c) proj = proj + row[c] * u[c];
    for (int c = 0; c < d; ++c) row[c] = (row[c] - proj * u[c]) + a_sink * u[c];
  } else {
    for (int c = 0; c < d; ++c)
      row[c] = a_hh * u[c] + 0.3 * normal12(key, (uint32_t)(p * d + c), sid, K_HHNOISE);
  }
}

SY_HD int hh_slot(const synth_spec& sp) {
  return sp.hh_count > 0 ? (sp.hh_hi - sp.hh_lo) / sp.hh_count : 0;
}

// 0 = plain row, 1 = sink, 2 = heavy hitter.
SY_HD int row_kind(const synth_spec& sp, int p, const int32_t* starts) {
  if (p < sp.n_sinks) return 1;
  if (sp.hh_count > 0 && p >= sp.hh_lo) {
    const int slot = hh_slot(sp);
    const int s = (p - sp.hh_lo) / slot;
    if (s < sp.hh_count && p >= starts[s] && p < starts[s] + sp.hh_span) return 2;
  }
  return 0;
}

void outliers_for(const synth_spec& sp, int layer, int b, int kvh, int32_t* ch) {
  const Key key = seq_key(sp.seed, sp.seq_stride, b);
  const uint32_t sid = stream_id(layer, b, kvh);
  int n = 0;
  for (uint32_t j = 0; n < sp.n_outlier && j < 4096; ++j) {
    const int c = (int)(draw_u32(key, j, sid, K_OUTL) % (uint32_t)sp.head_dim);
    if (!is_outlier(ch, n, c)) ch[n++] = c;
  }
}

void starts_for(const synth_spec& sp, int layer, int b, int kvh, int32_t* st) {
  const Key key = seq_key(sp.seed, sp.seq_stride, b);
  const uint32_t sid = stream_id(layer, b, kvh);
  const int slot = hh_slot(sp);
  for (int s = 0; s < sp.hh_count; ++s)
    st[s] = sp.hh_lo + s * slot +
            (int)(draw_u32(key, (uint32_t)s, sid, K_HHPOS) % (uint32_t)(slot - sp.hh_span + 1));
}

bool planting(const synth_spec& sp) { return sp.n_sinks > 0 || sp.hh_count > 0; }

// Unnormalised query-mean direction for (b, kv head): column sums over the group's window rows.
void dir_sums(const synth_spec& sp, const void* qwin, int b, int kvh, double* m) {
  const int d = sp.head_dim, G = sp.n_q_heads / sp.n_kv_heads;
  for (int c = 0; c < d; ++c) m[c] = 0.0;
  for (int g = 0; g < G; ++g) {
    const size_t base = ((size_t)b * sp.n_q_heads + (size_t)kvh * G + g) * sp.W * d;
    for (int t = 0; t < sp.W; ++t)
      for (int c = 0; c < d; ++c) m[c] = m[c] + load_elt(qwin, base + (size_t)t * d + c, sp.dtype);
  }
}

void normalise(int d, double* m) {
  double ss = 0.0;
  for (int c = 0; c < d; ++c) ss = ss + m[c] * m[c];
  if (ss == 0.0) {
    for (int c = 0; c < d; ++c) m[c] = c == 0 ? 1.0 : 0.0;
    return;
  }
  const double nrm = sqrt(ss);
  for (int c = 0; c < d; ++c) m[c] = m[c] / nrm;
}

// ---------------------------------------------------------------- device kernels
__global__ void k_qwin(synth_spec sp, int layer0, int n_layers, const double* rope, void* out) {
  const int d = sp.head_dim, half = d / 2;
  const size_t total = (size_t)n_layers * sp.batch * sp.n_q_heads * sp.W * half;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    size_t r = i / half;
    const int pr = (int)(i % half);
    const int t = (int)(r % sp.W);
    r /= sp.W;
    const int h = (int)(r % sp.n_q_heads);
    r /= sp.n_q_heads;
    const int b = (int)(r % sp.batch);
    const int l = (int)(r / sp.batch);
    const int p = sp.T - sp.W + t;
    const Key key = seq_key(sp.seed, sp.seq_stride, b);
    const uint32_t sid = stream_id(layer0 + l, b, h);
    const int c = 2 * pr;
    double x = normal12(key, (uint32_t)(p * d + c), sid, K_QWIN);
    double y = normal12(key, (uint32_t)(p * d + c + 1), sid, K_QWIN);
    if (sp.rope) rotate(&x, &y, rope + ((size_t)p * half + pr) * 2);
    const size_t o = (((size_t)l * sp.batch + b) * sp.n_q_heads + h) * sp.W * d + (size_t)t * d + c;
    store_elt(out, o, sp.dtype, x);
    store_elt(out, o + 1, sp.dtype, y);
  }
}

// Column sums of one layer's window queries per (b, kv head, channel), same order as the host.
__global__ void k_dir_sums(synth_spec sp, const void* qwin_layer, double* m) {
  const int d = sp.head_dim, G = sp.n_q_heads / sp.n_kv_heads;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= sp.batch * sp.n_kv_heads * d) return;
  const int c = i % d, kvh = (i / d) % sp.n_kv_heads, b = i / (d * sp.n_kv_heads);
  double acc = 0.0;
  for (int g = 0; g < G; ++g) {
    const size_t base = ((size_t)b * sp.n_q_heads + (size_t)kvh * G + g) * sp.W * d;
    for (int t = 0; t < sp.W; ++t) acc = acc + load_elt(qwin_layer, base + (size_t)t * d + c, sp.dtype);
  }
  m[i] = acc;
}

// Plain K pairs and all V pairs of one layer; planted K rows are left to k_planted.
__global__ void k_kv(synth_spec sp, int layer, int l_local, const double* rope,
                     const int32_t* outl, const int32_t* starts, void* k, void* v) {
  const int d = sp.head_dim, half = d / 2;
  const size_t total = (size_t)sp.batch * sp.n_kv_heads * sp.T * half;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    size_t r = i / half;
    const int pr = (int)(i % half);
    const int p = (int)(r % sp.T);
    r /= sp.T;
    const int h = (int)(r % sp.n_kv_heads);
    const int b = (int)(r / sp.n_kv_heads);
    const Key key = seq_key(sp.seed, sp.seq_stride, b);
    const uint32_t sid = stream_id(layer, b, h);
    const int c = 2 * pr;
    const size_t hb = (size_t)b * sp.n_kv_heads + h;
    const size_t o = (((size_t)l_local * sp.batch * sp.n_kv_heads) + hb) * sp.T * d + (size_t)p * d + c;
    const int32_t* st = starts + hb * (sp.hh_count > 0 ? sp.hh_count : 1);
    if (row_kind(sp, p, st) == 0) {
      double x, y;
      key_pair(sp, key, sid, p, c, outl + hb * (sp.n_outlier > 0 ? sp.n_outlier : 1), rope, &x, &y);
      store_elt(k, o, sp.dtype, x);
      store_elt(k, o + 1, sp.dtype, y);
    }
    store_elt(v, o, sp.dtype, normal12(key, (uint32_t)(p * d + c), sid, K_VAL));
    store_elt(v, o + 1, sp.dtype, normal12(key, (uint32_t)(p * d + c + 1), sid, K_VAL));
  }
}

__global__ void k_planted(synth_spec sp, int layer, int l_local, const double* rope,
                          const int32_t* outl, const int32_t* starts, const double* u,
                          double a_sink, double a_hh, void* k) {
  const int d = sp.head_dim;
  const int per_head = sp.n_sinks + sp.hh_count * sp.hh_span;
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= sp.batch * sp.n_kv_heads * per_head) return;
  const int r = i % per_head, hb = i / per_head;
  const int b = hb / sp.n_kv_heads, h = hb % sp.n_kv_heads;
  const int32_t* st = starts + (size_t)hb * (sp.hh_count > 0 ? sp.hh_count : 1);
  const int p = r < sp.n_sinks ? r : st[(r - sp.n_sinks) / sp.hh_span] + (r - sp.n_sinks) % sp.hh_span;
  const Key key = seq_key(sp.seed, sp.seq_stride, b);
  const uint32_t sid = stream_id(layer, b, h);
  double row[256];
  planted_row(sp, key, sid, p, r < sp.n_sinks, outl + (size_t)hb * (sp.n_outlier > 0 ? sp.n_outlier : 1),
              rope, u + (size_t)hb * d, a_sink, a_hh, row);
  const size_t o = (((size_t)l_local * sp.batch * sp.n_kv_heads) + hb) * sp.T * d + (size_t)p * d;
  for (int c = 0; c < d; ++c) store_elt(k, o + c, sp.dtype, row[c]);
}

__global__ void k_dq(synth_spec sp, int step, void* q) {
  const int d = sp.head_dim;
  const size_t total = (size_t)sp.n_layers * sp.batch * sp.n_q_heads * d;
  for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % d);
    size_t r = i / d;
    const int h = (int)(r % sp.n_q_heads);
    r /= sp.n_q_heads;
    const int b = (int)(r % sp.batch);
    const int l = (int)(r / sp.batch);
    const Key key = seq_key(sp.seed, sp.seq_stride, b);
    store_elt(q, i, sp.dtype, normal12(key, (uint32_t)(step * d + c), stream_id(l, b, h), K_DECQ));
  }
}

int grid_for(size_t total, int block) {
  size_t g = (total + block - 1) / block;
  if (g > 65536 * 8) g = 65536 * 8;
  return g ? (int)g : 1;
}

}  // namespace

// ---------------------------------------------------------------- host entry points
extern "C" int synth_validate(const synth_spec* sp) {
  if (!sp) return 1;
  if (sp->n_layers <= 0 || sp->batch <= 0 || sp->n_q_heads <= 0 || sp->n_kv_heads <= 0) return 1;
  if (sp->n_q_heads % sp->n_kv_heads) return 1;
  if (sp->head_dim < 2 || sp->head_dim > 256 || (sp->head_dim & 1)) return 1;
  if (sp->dtype < SYNTH_FP32 || sp->dtype > SYNTH_BF16) return 1;
  if (sp->T <= 0 || sp->W < 0 || sp->W > sp->T) return 1;
  if ((int64_t)sp->T * sp->head_dim >= (int64_t)1 << 31) return 1;
  if (sp->n_layers > 1024 || sp->n_q_heads > 1024 || sp->batch > 4096) return 1;
  if (sp->n_outlier < 0 || sp->n_outlier > 16 || sp->n_outlier > sp->head_dim / 2) return 1;
  if (sp->n_sinks < 0 || sp->n_sinks > sp->T) return 1;
  if (sp->hh_count < 0) return 1;
  if (sp->hh_count > 0) {
    if (sp->hh_span < 1 || sp->hh_lo < sp->n_sinks || sp->hh_hi > sp->T || sp->hh_hi <= sp->hh_lo)
      return 1;
    if ((sp->hh_hi - sp->hh_lo) / sp->hh_count < sp->hh_span) return 1;
  }
  if ((sp->n_sinks > 0 || sp->hh_count > 0) && sp->W == 0) return 1;
  return 0;
}

extern "C" int synth_rope_table(int32_t T, int32_t d, double base, double* out) {
  if (T <= 0 || d < 2 || (d & 1) || !out) return 1;
  const int half = d / 2;
  for (int i = 0; i < half; ++i) {
    const double inv = pow(base, -(2.0 * i) / (double)d);
    for (int p = 0; p < T; ++p) {
      const double a = (double)p * inv;
      out[((size_t)p * half + i) * 2] = cos(a);
      out[((size_t)p * half + i) * 2 + 1] = sin(a);
    }
  }
  return 0;
}

extern "C" int synth_outlier_channels(const synth_spec* sp, int32_t layer, int32_t b, int32_t kvh,
                                      int32_t* ch) {
  if (synth_validate(sp) || !ch) return 1;
  outliers_for(*sp, layer, b, kvh, ch);
  return 0;
}

extern "C" int synth_hh_starts(const synth_spec* sp, int32_t layer, int32_t b, int32_t kvh,
                               int32_t* starts) {
  if (synth_validate(sp) || !starts) return 1;
  starts_for(*sp, layer, b, kvh, starts);
  return 0;
}

extern "C" int synth_qwin_host(const synth_spec* sp, int32_t layer, const double* rope, void* out) {
  if (synth_validate(sp) || !out || (sp->rope && !rope)) return 1;
  const int d = sp->head_dim;
  const int64_t rows = (int64_t)sp->batch * sp->n_q_heads * sp->W;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const int t = (int)(r % sp->W);
    const int h = (int)((r / sp->W) % sp->n_q_heads);
    const int b = (int)(r / ((int64_t)sp->W * sp->n_q_heads));
    qwin_row(*sp, layer, b, h, sp->T - sp->W + t, rope, out, (size_t)r * d);
  }
  return 0;
}

extern "C" int synth_unit_dir_host(const synth_spec* sp, const void* qwin_layer, double* u) {
  if (synth_validate(sp) || !qwin_layer || !u || sp->W == 0) return 1;
  const int d = sp->head_dim;
  for (int b = 0; b < sp->batch; ++b)
    for (int h = 0; h < sp->n_kv_heads; ++h) {
      double* m = u + ((size_t)b * sp->n_kv_heads + h) * d;
      dir_sums(*sp, qwin_layer, b, h, m);
      normalise(d, m);
    }
  return 0;
}

extern "C" int synth_kv_host(const synth_spec* sp, int32_t layer, const void* qwin_layer,
                             const double* rope, void* k, void* v) {
  if (synth_validate(sp) || !k || !v || (sp->rope && !rope)) return 1;
  if (planting(*sp) && !qwin_layer) return 1;
  const int d = sp->head_dim, H = sp->n_kv_heads;
  const double a_sink = 4.0 * sqrt((double)d), a_hh = 3.0 * sqrt((double)d);
  const int nh = sp->batch * H;
  double* u = (double*)calloc((size_t)nh * d, sizeof(double));
  int32_t* outl = (int32_t*)calloc((size_t)nh * (sp->n_outlier + 1), sizeof(int32_t));
  int32_t* st = (int32_t*)calloc((size_t)nh * (sp->hh_count + 1), sizeof(int32_t));
  if (!u || !outl || !st) {
    free(u); free(outl); free(st);
    return 2;
  }
  if (planting(*sp)) synth_unit_dir_host(sp, qwin_layer, u);
  for (int hb = 0; hb < nh; ++hb) {
    outliers_for(*sp, layer, hb / H, hb % H, outl + (size_t)hb * (sp->n_outlier + 1));
    starts_for(*sp, layer, hb / H, hb % H, st + (size_t)hb * (sp->hh_count + 1));
  }
  const int64_t rows = (int64_t)nh * sp->T;
#pragma omp parallel for schedule(static)
  for (int64_t r = 0; r < rows; ++r) {
    const int p = (int)(r % sp->T);
    const int hb = (int)(r / sp->T);
    const int b = hb / H, h = hb % H;
    const Key key = seq_key(sp->seed, sp->seq_stride, b);
    const uint32_t sid = stream_id(layer, b, h);
    const int32_t* ol = outl + (size_t)hb * (sp->n_outlier + 1);
    const int kind = row_kind(*sp, p, st + (size_t)hb * (sp->hh_count + 1));
    const size_t o = (size_t)r * d;
    if (kind == 0) {
      for (int c = 0; c < d; c += 2) {
        double x, y;
        key_pair(*sp, key, sid, p, c, ol, rope, &x, &y);
        store_elt(k, o + c, sp->dtype, x);
        store_elt(k, o + c + 1, sp->dtype, y);
      }
    } else {
      double row[256];
      planted_row(*sp, key, sid, p, kind == 1, ol, rope, u + (size_t)hb * d, a_sink, a_hh, row);
      for (int c = 0; c < d; ++c) store_elt(k, o + c, sp->dtype, row[c]);
    }
    for (int c = 0; c < d; ++c)
      store_elt(v, o + c, sp->dtype, normal12(key, (uint32_t)(p * d + c), sid, K_VAL));
  }
  free(u);
  free(outl);
  free(st);
  return 0;
}

extern "C" int synth_dq_host(const synth_spec* sp, int32_t step, void* q) {
  if (synth_validate(sp) || !q || step < 0) return 1;
  const int d = sp->head_dim;
  const int64_t total = (int64_t)sp->n_layers * sp->batch * sp->n_q_heads * d;
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < total; ++i) {
    const int c = (int)(i % d);
    int64_t r = i / d;
    const int h = (int)(r % sp->n_q_heads);
    r /= sp->n_q_heads;
    const int b = (int)(r % sp->batch);
    const int l = (int)(r / sp->batch);
    store_elt(q, (size_t)i, sp->dtype,
              normal12(seq_key(sp->seed, sp->seq_stride, b), (uint32_t)(step * d + c),
                       stream_id(l, b, h), K_DECQ));
  }
  return 0;
}

// ---------------------------------------------------------------- device entry points
extern "C" int synth_qwin_dev(const synth_spec* sp, int32_t layer0, int32_t n_layers,
                              const double* rope_dev, void* out, void* stream) {
  if (synth_validate(sp) || !out || (sp->rope && !rope_dev) || n_layers <= 0) return 1;
  if (sp->W == 0) return 0;
  const size_t total = (size_t)n_layers * sp->batch * sp->n_q_heads * sp->W * (sp->head_dim / 2);
  hipLaunchKernelGGL(k_qwin, dim3(grid_for(total, 256)), dim3(256), 0, (hipStream_t)stream, *sp,
                     layer0, n_layers, rope_dev, out);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}

// Generates K and V for layers [layer0, layer0 + n_layers) into [n_layers][B][Hkv][T][d].
// When planting is on, the query-mean direction of each layer is reduced on the device and
// normalised on the host (same routine as the host path); this call synchronises `stream`.
extern "C" int synth_kv_dev(const synth_spec* sp, int32_t layer0, int32_t n_layers,
                            const void* qwin_dev, const double* rope_dev, double* u_ws, void* k,
                            void* v, void* stream) {
  if (synth_validate(sp) || !k || !v || (sp->rope && !rope_dev) || n_layers <= 0) return 1;
  if (planting(*sp) && (!qwin_dev || !u_ws)) return 1;
  hipStream_t st = (hipStream_t)stream;
  const int d = sp->head_dim, H = sp->n_kv_heads, nh = sp->batch * H;
  const int no = sp->n_outlier > 0 ? sp->n_outlier : 1, nc = sp->hh_count > 0 ? sp->hh_count : 1;
  int32_t* h_outl = (int32_t*)calloc((size_t)nh * no, sizeof(int32_t));
  int32_t* h_st = (int32_t*)calloc((size_t)nh * nc, sizeof(int32_t));
  double* h_u = (double*)calloc((size_t)nh * d, sizeof(double));
  int32_t *d_outl = nullptr, *d_st = nullptr;
  int rc = 0;
  if (!h_outl || !h_st || !h_u) rc = 2;
  if (!rc && hipMalloc((void**)&d_outl, (size_t)nh * no * sizeof(int32_t)) != hipSuccess) rc = 3;
  if (!rc && hipMalloc((void**)&d_st, (size_t)nh * nc * sizeof(int32_t)) != hipSuccess) rc = 3;
  const double a_sink = 4.0 * sqrt((double)d), a_hh = 3.0 * sqrt((double)d);
  const size_t qwin_layer = (size_t)sp->batch * sp->n_q_heads * sp->W * d;
  const size_t elt = sp->dtype == SYNTH_FP32 ? 4 : 2;
  for (int l = 0; l < n_layers && !rc; ++l) {
    const int layer = layer0 + l;
    for (int hb = 0; hb < nh; ++hb) {
      if (sp->n_outlier > 0) outliers_for(*sp, layer, hb / H, hb % H, h_outl + (size_t)hb * no);
      if (sp->hh_count > 0) starts_for(*sp, layer, hb / H, hb % H, h_st + (size_t)hb * nc);
    }
    if (hipMemcpyAsync(d_outl, h_outl, (size_t)nh * no * 4, hipMemcpyHostToDevice, st) != hipSuccess ||
        hipMemcpyAsync(d_st, h_st, (size_t)nh * nc * 4, hipMemcpyHostToDevice, st) != hipSuccess) {
      rc = 3;
      break;
    }
    const size_t total = (size_t)nh * sp->T * (d / 2);
    hipLaunchKernelGGL(k_kv, dim3(grid_for(total, 256)), dim3(256), 0, st, *sp, layer, l, rope_dev,
                       d_outl, d_st, k, v);
    if (planting(*sp)) {
      const void* ql = (const char*)qwin_dev + (size_t)l * qwin_layer * elt;
      hipLaunchKernelGGL(k_dir_sums, dim3((nh * d + 255) / 256), dim3(256), 0, st, *sp, ql, u_ws);
      if (hipMemcpyAsync(h_u, u_ws, (size_t)nh * d * 8, hipMemcpyDeviceToHost, st) != hipSuccess ||
          hipStreamSynchronize(st) != hipSuccess) {
        rc = 3;
        break;
      }
      for (int hb = 0; hb < nh; ++hb) normalise(d, h_u + (size_t)hb * d);
      if (hipMemcpyAsync(u_ws, h_u, (size_t)nh * d * 8, hipMemcpyHostToDevice, st) != hipSuccess) {
        rc = 3;
        break;
      }
      const int per_head = sp->n_sinks + sp->hh_count * sp->hh_span;
      hipLaunchKernelGGL(k_planted, dim3((nh * per_head + 63) / 64), dim3(64), 0, st, *sp, layer, l,
                         rope_dev, d_outl, d_st, u_ws, a_sink, a_hh, k);
    }
    // the per-layer host tables are reused next iteration
    if (hipStreamSynchronize(st) != hipSuccess) rc = 3;
  }
  if (hipGetLastError() != hipSuccess && !rc) rc = 3;
  if (d_outl) (void)hipFree(d_outl);
  if (d_st) (void)hipFree(d_st);
  free(h_outl);
  free(h_st);
  free(h_u);
  return rc;
}

extern "C" int synth_dq_dev(const synth_spec* sp, int32_t step, void* q, void* stream) {
  if (synth_validate(sp) || !q || step < 0) return 1;
  const size_t total = (size_t)sp->n_layers * sp->batch * sp->n_q_heads * sp->head_dim;
  hipLaunchKernelGGL(k_dq, dim3(grid_for(total, 256)), dim3(256), 0, (hipStream_t)stream, *sp, step, q);
  return hipGetLastError() == hipSuccess ? 0 : 3;
}
