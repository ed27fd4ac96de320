/*
 * Oracle for the multi-DNN inference hot path of D-STACK (arxiv 2304.13541).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the tests, the smoke check and the CPU-baseline leg of
 * the benchmark do.  It shares no code, header or table with the HIP library.
 *
 * What it computes: the plain definition of each network's forward pass in
 * fp64 -- direct cross-correlation convolution, depthwise convolution, naive
 * matrix products, max/average pooling, inference-mode batch norm, ReLU /
 * ReLU6 and the LSTM cell, and for the transformer layer normalisation,
 * scaled dot-product self-attention with a softmax, GELU and tanh -- over
 * the architectures the paper evaluates or the workloads name: a tiny 4-conv
 * CNN, ResNet-50 (v1.5), MobileNetV2, VGG-19, a 2-layer LSTM and a
 * BERT-base encoder (Sec. 4.4's transformer, 10- and 20-word sentences).  The paper itself runs stock framework kernels
 * (Sec. 3, Sec. 4.1 and its A.int table); the layers' mathematics is the
 * textbook one, written out here loop by loop.
 *
 * Storage points ("parity" mode): the GPU path stores activations as bf16
 * between layers, so in parity mode every layer output that the GPU stores
 * as bf16 is rounded to bf16 (round-to-nearest-even) at the same point.  In
 * pure mode nothing is rounded after the bf16 inputs and weights.
 *
 * Weights come from an independent implementation of the weight-generation
 * rule (splitmix64 streams, Box-Muller normals, bf16 RNE), written from the
 * published definitions of those algorithms:
 *   splitmix64: Steele, Lea, Flood, "Fast splittable pseudorandom number
 *   generators", OOPSLA 2014 (constants as in Vigna's reference code);
 *   Box-Muller: Box & Muller, Ann. Math. Statist. 29 (1958).
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* bf16 helpers                                                        */
/* ------------------------------------------------------------------ */

/* Round x to the nearest bf16 value (8 significant bits), ties to even,
 * done on the real value: scale by a power of two so that the bf16 quantum
 * becomes 1, round with nearbyint (default mode = nearest-even), scale back. */
double oracle_bf16_round(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  frexp(x, &e);            /* |x| = f * 2^e with f in [0.5, 1) */
  int qe = e - 8;          /* quantum of an 8-significant-bit number */
  if (qe < -133) qe = -133; /* bf16 subnormal quantum is 2^-133 */
  return ldexp(nearbyint(ldexp(x, -qe)), qe);
}

static uint16_t to_bf16_bits(double x) {
  float f = (float)oracle_bf16_round(x); /* exact: value has <= 8 significant bits */
  uint32_t u;
  memcpy(&u, &f, 4);
  return (uint16_t)(u >> 16);
}

double oracle_bf16_to_double(uint16_t h) {
  uint32_t u = (uint32_t)h << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* ------------------------------------------------------------------ */
/* weight generation                                                   */
/* ------------------------------------------------------------------ */

static uint64_t sm64_next(uint64_t* state) {
  uint64_t z = (*state += 0x9E3779B97F4A7C15ULL);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}

/* uniform in (0, 1]: 53 random bits scaled by 2^-53, with 0 replaced by 1 */
static double sm64_unit(uint64_t* state) {
  double u = (double)(sm64_next(state) >> 11) * 0x1.0p-53;
  return u == 0.0 ? 1.0 : u;
}

static uint64_t stream_init(uint64_t seed, int tensor_index) {
  return seed ^ (0x9E3779B97F4A7C15ULL * (uint64_t)(tensor_index + 1));
}

/* N(0, std^2) values, Box-Muller pairs in order, rounded to bf16 */
static void gen_normal(uint64_t seed, int idx, double std, double* out, long n) {
  uint64_t st = stream_init(seed, idx);
  const double two_pi = 6.283185307179586; /* 2*pi rounded to fp64 */
  for (long i = 0; i < n; i += 2) {
    double u1 = sm64_unit(&st);
    double u2 = sm64_unit(&st);
    double r = sqrt(-2.0 * log(u1));
    double a = two_pi * u2;
    double z0 = r * cos(a);
    double z1 = r * sin(a);
    out[i] = oracle_bf16_round(z0 * std);
    if (i + 1 < n) out[i + 1] = oracle_bf16_round(z1 * std);
  }
}

/* U(-a, a] values: (2u - 1) * a, rounded to bf16 */
static void gen_uniform(uint64_t seed, int idx, double a, double* out, long n) {
  uint64_t st = stream_init(seed, idx);
  for (long i = 0; i < n; ++i) {
    double u = sm64_unit(&st);
    double t = 2.0 * u;
    t = t - 1.0;
    out[i] = oracle_bf16_round(t * a);
  }
}

/* ------------------------------------------------------------------ */
/* layer primitives (fp64, plain loops)                                */
/* ------------------------------------------------------------------ */

static int out_dim(int in, int k, int stride, int pad) { return (in + 2 * pad - k) / stride + 1; }

/* Convolution, groups = 1, cross-correlation (no kernel flip).
 * x: [N][H][W][C], w: [K][R][S][C], y: [N][Ho][Wo][K].
 * y[n,ho,wo,k] = sum_{r,s,c} x[n, ho*st - pad + r, wo*st - pad + s, c] * w[k,r,s,c],
 * with x taken as zero outside the image. */
void oracle_conv2d(const double* x, int N, int H, int W, int C, const double* w, int K, int R, int S,
                   int stride, int pad, double* y) {
  int Ho = out_dim(H, R, stride, pad), Wo = out_dim(W, S, stride, pad);
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int ho = 0; ho < Ho; ++ho)
      for (int wo = 0; wo < Wo; ++wo)
        for (int k = 0; k < K; ++k) {
          double acc = 0.0;
          for (int r = 0; r < R; ++r) {
            int hi = ho * stride - pad + r;
            if (hi < 0 || hi >= H) continue;
            for (int s = 0; s < S; ++s) {
              int wi = wo * stride - pad + s;
              if (wi < 0 || wi >= W) continue;
              const double* xp = x + (((long)n * H + hi) * W + wi) * C;
              const double* wp = w + (((long)k * R + r) * S + s) * C;
              for (int c = 0; c < C; ++c) acc += xp[c] * wp[c];
            }
          }
          y[(((long)n * Ho + ho) * Wo + wo) * K + k] = acc;
        }
}

/* Depthwise 3x3-style convolution: one filter per channel.
 * x: [N][H][W][C], w: [C][R][S], y: [N][Ho][Wo][C]. */
void oracle_dwconv(const double* x, int N, int H, int W, int C, const double* w, int R, int S, int stride,
                   int pad, double* y) {
  int Ho = out_dim(H, R, stride, pad), Wo = out_dim(W, S, stride, pad);
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int ho = 0; ho < Ho; ++ho)
      for (int wo = 0; wo < Wo; ++wo)
        for (int c = 0; c < C; ++c) {
          double acc = 0.0;
          for (int r = 0; r < R; ++r) {
            int hi = ho * stride - pad + r;
            if (hi < 0 || hi >= H) continue;
            for (int s = 0; s < S; ++s) {
              int wi = wo * stride - pad + s;
              if (wi < 0 || wi >= W) continue;
              acc += x[(((long)n * H + hi) * W + wi) * C + c] * w[((long)c * R + r) * S + s];
            }
          }
          y[(((long)n * Ho + ho) * Wo + wo) * C + c] = acc;
        }
}

/* Fully connected: y[b][o] = sum_i x[b][i] * w[o][i] + bias[o]  (w: [O][I]) */
void oracle_fc(const double* x, int B, int I, const double* w, const double* bias, int O, double* y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < B; ++b)
    for (int o = 0; o < O; ++o) {
      double acc = 0.0;
      for (int i = 0; i < I; ++i) acc += x[(long)b * I + i] * w[(long)o * I + i];
      y[(long)b * O + o] = acc + (bias ? bias[o] : 0.0);
    }
}

/* Max pooling, window k x k, given stride and pad; padded cells never win. */
void oracle_maxpool(const double* x, int N, int H, int W, int C, int k, int stride, int pad, double* y) {
  int Ho = out_dim(H, k, stride, pad), Wo = out_dim(W, k, stride, pad);
  for (int n = 0; n < N; ++n)
    for (int ho = 0; ho < Ho; ++ho)
      for (int wo = 0; wo < Wo; ++wo)
        for (int c = 0; c < C; ++c) {
          double m = -INFINITY;
          for (int r = 0; r < k; ++r) {
            int hi = ho * stride - pad + r;
            if (hi < 0 || hi >= H) continue;
            for (int s = 0; s < k; ++s) {
              int wi = wo * stride - pad + s;
              if (wi < 0 || wi >= W) continue;
              double v = x[(((long)n * H + hi) * W + wi) * C + c];
              if (v > m) m = v;
            }
          }
          y[(((long)n * Ho + ho) * Wo + wo) * C + c] = m;
        }
}

/* Global average pooling: y[n][c] = mean over H x W of x[n,:,:,c] */
void oracle_avgpool(const double* x, int N, int H, int W, int C, double* y) {
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c) {
      double s = 0.0;
      for (int i = 0; i < H * W; ++i) s += x[((long)n * H * W + i) * C + c];
      y[(long)n * C + c] = s / (double)(H * W);
    }
}

/* Inference batch norm on the last axis: z = gamma*(y - mean)/sqrt(var + eps) + beta */
static void batchnorm(double* y, long rows, int C, const double* gamma, const double* beta, const double* mean,
                      const double* var, double eps) {
  for (long i = 0; i < rows; ++i)
    for (int c = 0; c < C; ++c) {
      double v = y[i * C + c];
      y[i * C + c] = gamma[c] * (v - mean[c]) / sqrt(var[c] + eps) + beta[c];
    }
}

static double sigmoid(double v) { return 1.0 / (1.0 + exp(-v)); }

/* One LSTM layer over a sequence (gate order i, f, g, o; h0 = c0 = 0).
 * x: [T][B][I]; w_ih: [4H][I]; w_hh: [4H][H]; b_ih, b_hh: [4H]; h_out: [T][B][H].
 * gates = W_ih x_t + b_ih + W_hh h_{t-1} + b_hh; i,f,o = sigmoid, g = tanh;
 * c_t = f*c_{t-1} + i*g; h_t = o*tanh(c_t).
 * round_h_for_gemm: h_{t-1} is rounded to bf16 where it enters the product. */
void oracle_lstm_layer(const double* x, int T, int B, int I, int Hd, const double* w_ih, const double* w_hh,
                       const double* b_ih, const double* b_hh, int round_h_for_gemm, double* h_out, double* c_last) {
  double* h = calloc((size_t)B * Hd, sizeof(double));
  double* hq = calloc((size_t)B * Hd, sizeof(double));
  double* c = calloc((size_t)B * Hd, sizeof(double));
  double* g = malloc(sizeof(double) * (size_t)B * 4 * Hd);
  for (int t = 0; t < T; ++t) {
    for (long i = 0; i < (long)B * Hd; ++i) hq[i] = round_h_for_gemm ? oracle_bf16_round(h[i]) : h[i];
#pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b)
      for (int j = 0; j < 4 * Hd; ++j) {
        const double* xt = x + ((long)t * B + b) * I;
        double acc = b_ih[j] + b_hh[j];
        for (int i = 0; i < I; ++i) acc += w_ih[(long)j * I + i] * xt[i];
        for (int k = 0; k < Hd; ++k) acc += w_hh[(long)j * Hd + k] * hq[(long)b * Hd + k];
        g[(long)b * 4 * Hd + j] = acc;
      }
    for (int b = 0; b < B; ++b)
      for (int k = 0; k < Hd; ++k) {
        const double* gb = g + (long)b * 4 * Hd;
        double ig = sigmoid(gb[k]);
        double fg = sigmoid(gb[Hd + k]);
        double gg = tanh(gb[2 * Hd + k]);
        double og = sigmoid(gb[3 * Hd + k]);
        double cn = fg * c[(long)b * Hd + k] + ig * gg;
        c[(long)b * Hd + k] = cn;
        h[(long)b * Hd + k] = og * tanh(cn);
        h_out[((long)t * B + b) * Hd + k] = h[(long)b * Hd + k];
      }
  }
  if (c_last) memcpy(c_last, c, sizeof(double) * (size_t)B * Hd);
  free(h);
  free(hq);
  free(c);
  free(g);
}

/* Layer normalisation of each of `rows` rows of C values:
 * y = (x - mean) / sqrt(var + eps) * gamma + beta, mean and (biased)
 * variance over the row. */
void oracle_layernorm(const double* x, long rows, int C, const double* gamma, const double* beta, double eps,
                      double* y) {
  for (long r = 0; r < rows; ++r) {
    const double* xr = x + r * C;
    double mean = 0.0;
    for (int c = 0; c < C; ++c) mean += xr[c];
    mean /= C;
    double var = 0.0;
    for (int c = 0; c < C; ++c) var += (xr[c] - mean) * (xr[c] - mean);
    var /= C;
    const double inv = 1.0 / sqrt(var + eps);
    for (int c = 0; c < C; ++c) y[r * C + c] = (xr[c] - mean) * inv * gamma[c] + beta[c];
  }
}

/* Multi-head self-attention core of one batch of B sequences of T tokens:
 * qkv [B][T][3*Hm] holds per token the queries, keys and values (each Hm =
 * heads * dh wide, head h at columns h*dh..); for every sequence and head,
 * s[i][j] = q_i . k_j / sqrt(dh), p = softmax over j, o_i = sum_j p[i][j] v_j
 * written to out [B][T][Hm] at the head's columns.  No mask. */
void oracle_attention(const double* qkv, int B, int T, int heads, int dh, double* out) {
  const int Hm = heads * dh;
  double* s = malloc(sizeof(double) * (size_t)T);
  for (int b = 0; b < B; ++b)
    for (int h = 0; h < heads; ++h)
      for (int i = 0; i < T; ++i) {
        const double* q = qkv + ((long)b * T + i) * 3 * Hm + h * dh;
        double mx = -INFINITY;
        for (int j = 0; j < T; ++j) {
          const double* k = qkv + ((long)b * T + j) * 3 * Hm + Hm + h * dh;
          double d = 0.0;
          for (int e = 0; e < dh; ++e) d += q[e] * k[e];
          s[j] = d / sqrt((double)dh);
          if (s[j] > mx) mx = s[j];
        }
        double sum = 0.0;
        for (int j = 0; j < T; ++j) {
          s[j] = exp(s[j] - mx);
          sum += s[j];
        }
        double* o = out + ((long)b * T + i) * Hm + h * dh;
        for (int e = 0; e < dh; ++e) {
          double a = 0.0;
          for (int j = 0; j < T; ++j) a += s[j] / sum * qkv[((long)b * T + j) * 3 * Hm + 2 * Hm + h * dh + e];
          o[e] = a;
        }
      }
  free(s);
}

/* ------------------------------------------------------------------ */
/* models                                                              */
/* ------------------------------------------------------------------ */

enum { ARCH_TINY = 0, ARCH_R50 = 1, ARCH_MBV2 = 2, ARCH_VGG = 3, ARCH_LSTM = 4, ARCH_BERT = 5, ARCH_BERT_LONG = 6 };
enum { DIST_HE = 0, DIST_ZERO = 1, DIST_UNIF = 2 };

typedef struct {
  long numel;
  int dist;
  int fan_in;
  double* v;
} tensor_t;

typedef struct {
  int arch;
  uint64_t seed;
  int nt, cap;
  tensor_t* t;
  int cursor; /* forward-pass read position */
} model_t;

static void add_tensor(model_t* m, long numel, int dist, int fan_in) {
  if (m->nt == m->cap) {
    m->cap = m->cap ? 2 * m->cap : 64;
    m->t = realloc(m->t, sizeof(tensor_t) * (size_t)m->cap);
  }
  tensor_t* t = &m->t[m->nt];
  t->numel = numel;
  t->dist = dist;
  t->fan_in = fan_in;
  t->v = malloc(sizeof(double) * (size_t)numel);
  if (dist == DIST_HE)
    gen_normal(m->seed, m->nt, sqrt(2.0 / (double)fan_in), t->v, numel);
  else if (dist == DIST_UNIF)
    gen_uniform(m->seed, m->nt, 1.0 / 32.0, t->v, numel);
  else
    memset(t->v, 0, sizeof(double) * (size_t)numel);
  m->nt++;
}

static const double* next_tensor(model_t* m) { return m->t[m->cursor++].v; }

/* ResNet-50 stage table: (blocks, bottleneck width, stride of the first block) */
static const int R50_STAGES[4][3] = {{3, 64, 1}, {4, 128, 2}, {6, 256, 2}, {3, 512, 2}};
/* MobileNetV2 inverted-residual table (t, c, n, s) */
static const int MBV2_CFG[7][4] = {{1, 16, 1, 1}, {6, 24, 2, 2}, {6, 32, 3, 2}, {6, 64, 4, 2},
                                   {6, 96, 3, 1}, {6, 160, 3, 2}, {6, 320, 1, 1}};
/* VGG-19 conv channels per stage (5 stages of 2/2/4/4/4 convs) */
static const int VGG_STAGE_CONVS[5] = {2, 2, 4, 4, 4};
static const int VGG_STAGE_CH[5] = {64, 128, 256, 512, 512};
/* BERT-base: 12 layers, width 768, 12 heads of 64, feed-forward 3072,
 * WordPiece vocabulary 30522, 512 positions, 2 token types, 2 classes.
 * Weights and biases N(0, 0.02^2) (the normal rule with fan-in 5000:
 * sqrt(2 / 5000) = 0.02); layer-norm gain 1 and bias 0 (constants, like the
 * CNNs' BN statistics); eps 1e-12. */
enum { BERT_L = 12, BERT_H = 768, BERT_HEADS = 12, BERT_DH = 64, BERT_FF = 3072, BERT_VOCAB = 30522,
       BERT_POS = 512, BERT_CLASSES = 2, BERT_FAN = 5000 };

static void build_tensors(model_t* m) {
  switch (m->arch) {
    case ARCH_TINY: {
      int ch[5] = {3, 16, 32, 32, 64};
      for (int l = 0; l < 4; ++l) add_tensor(m, (long)ch[l + 1] * 9 * ch[l], DIST_HE, 9 * ch[l]);
      add_tensor(m, 10L * 64, DIST_HE, 64);
      add_tensor(m, 10, DIST_ZERO, 0);
      break;
    }
    case ARCH_R50: {
      add_tensor(m, 64L * 49 * 3, DIST_HE, 49 * 3);
      int cin = 64;
      for (int st = 0; st < 4; ++st) {
        int planes = R50_STAGES[st][1], cout = 4 * planes;
        for (int b = 0; b < R50_STAGES[st][0]; ++b) {
          add_tensor(m, (long)planes * cin, DIST_HE, cin);              /* conv1 1x1 */
          add_tensor(m, (long)planes * 9 * planes, DIST_HE, 9 * planes); /* conv2 3x3 */
          add_tensor(m, (long)cout * planes, DIST_HE, planes);          /* conv3 1x1 */
          if (b == 0) add_tensor(m, (long)cout * cin, DIST_HE, cin);     /* downsample 1x1 */
          cin = cout;
        }
      }
      add_tensor(m, 1000L * 2048, DIST_HE, 2048);
      add_tensor(m, 1000, DIST_ZERO, 0);
      break;
    }
    case ARCH_MBV2: {
      add_tensor(m, 32L * 9 * 3, DIST_HE, 27);
      int cin = 32;
      for (int g = 0; g < 7; ++g) {
        int t = MBV2_CFG[g][0], c = MBV2_CFG[g][1], n = MBV2_CFG[g][2];
        for (int i = 0; i < n; ++i) {
          int hid = cin * t;
          if (t != 1) add_tensor(m, (long)hid * cin, DIST_HE, cin); /* expand 1x1 */
          add_tensor(m, (long)hid * 9, DIST_HE, 9);                 /* depthwise 3x3 */
          add_tensor(m, (long)c * hid, DIST_HE, hid);               /* project 1x1 */
          cin = c;
        }
      }
      add_tensor(m, 1280L * 320, DIST_HE, 320);
      add_tensor(m, 1000L * 1280, DIST_HE, 1280);
      add_tensor(m, 1000, DIST_ZERO, 0);
      break;
    }
    case ARCH_VGG: {
      int cin = 3;
      for (int st = 0; st < 5; ++st)
        for (int i = 0; i < VGG_STAGE_CONVS[st]; ++i) {
          int cout = VGG_STAGE_CH[st];
          add_tensor(m, (long)cout * 9 * cin, DIST_HE, 9 * cin);
          add_tensor(m, cout, DIST_ZERO, 0);
          cin = cout;
        }
      add_tensor(m, 4096L * 25088, DIST_HE, 25088);
      add_tensor(m, 4096, DIST_ZERO, 0);
      add_tensor(m, 4096L * 4096, DIST_HE, 4096);
      add_tensor(m, 4096, DIST_ZERO, 0);
      add_tensor(m, 1000L * 4096, DIST_HE, 4096);
      add_tensor(m, 1000, DIST_ZERO, 0);
      break;
    }
    case ARCH_LSTM: {
      int in = 512;
      for (int l = 0; l < 2; ++l) {
        add_tensor(m, 4096L * in, DIST_UNIF, 0);
        add_tensor(m, 4096L * 1024, DIST_UNIF, 0);
        add_tensor(m, 4096, DIST_UNIF, 0);
        add_tensor(m, 4096, DIST_UNIF, 0);
        in = 1024;
      }
      break;
    }
    case ARCH_BERT:
    case ARCH_BERT_LONG: {
      add_tensor(m, (long)BERT_VOCAB * BERT_H, DIST_HE, BERT_FAN); /* word embeddings */
      add_tensor(m, (long)BERT_POS * BERT_H, DIST_HE, BERT_FAN);   /* position embeddings */
      add_tensor(m, 2L * BERT_H, DIST_HE, BERT_FAN);               /* token-type embeddings */
      for (int l = 0; l < BERT_L; ++l) {
        add_tensor(m, 3L * BERT_H * BERT_H, DIST_HE, BERT_FAN); /* W_qkv [3H][H] (q, k, v rows) */
        add_tensor(m, 3L * BERT_H, DIST_HE, BERT_FAN);
        add_tensor(m, (long)BERT_H * BERT_H, DIST_HE, BERT_FAN); /* attention output */
        add_tensor(m, BERT_H, DIST_HE, BERT_FAN);
        add_tensor(m, (long)BERT_FF * BERT_H, DIST_HE, BERT_FAN); /* feed-forward in */
        add_tensor(m, BERT_FF, DIST_HE, BERT_FAN);
        add_tensor(m, (long)BERT_H * BERT_FF, DIST_HE, BERT_FAN); /* feed-forward out */
        add_tensor(m, BERT_H, DIST_HE, BERT_FAN);
      }
      add_tensor(m, (long)BERT_H * BERT_H, DIST_HE, BERT_FAN); /* pooler */
      add_tensor(m, BERT_H, DIST_HE, BERT_FAN);
      add_tensor(m, (long)BERT_CLASSES * BERT_H, DIST_HE, BERT_FAN); /* classifier */
      add_tensor(m, BERT_CLASSES, DIST_HE, BERT_FAN);
      break;
    }
  }
}

static int arch_id(const char* a) {
  if (!strcmp(a, "tinycnn")) return ARCH_TINY;
  if (!strcmp(a, "resnet50")) return ARCH_R50;
  if (!strcmp(a, "mobilenetv2")) return ARCH_MBV2;
  if (!strcmp(a, "vgg19")) return ARCH_VGG;
  if (!strcmp(a, "lstm2")) return ARCH_LSTM;
  if (!strcmp(a, "bert")) return ARCH_BERT;
  if (!strcmp(a, "bert_long")) return ARCH_BERT_LONG;
  return -1;
}

void* oracle_model_load(const char* arch, uint64_t seed) {
  int a = arch_id(arch);
  if (a < 0) return NULL;
  model_t* m = calloc(1, sizeof(model_t));
  m->arch = a;
  m->seed = seed;
  build_tensors(m);
  return m;
}

void oracle_model_free(void* h) {
  model_t* m = h;
  if (!m) return;
  for (int i = 0; i < m->nt; ++i) free(m->t[i].v);
  free(m->t);
  free(m);
}

/* test hook: overwrite tensor i with given values (planted weights) */
int oracle_model_set_tensor(void* h, int i, const double* v) {
  model_t* m = h;
  if (i < 0 || i >= m->nt) return -1;
  memcpy(m->t[i].v, v, sizeof(double) * (size_t)m->t[i].numel);
  return 0;
}

/* test hook: first n outputs of splitmix64 from a given state */
void oracle_splitmix64(uint64_t state, int n, uint64_t* out) {
  for (int i = 0; i < n; ++i) out[i] = sm64_next(&state);
}

int oracle_model_num_tensors(void* h) { return ((model_t*)h)->nt; }
long oracle_model_tensor_numel(void* h, int i) { return ((model_t*)h)->t[i].numel; }

/* bf16 bit patterns of tensor i, in its logical element order */
int oracle_model_tensor_bf16(void* h, int i, uint16_t* out) {
  model_t* m = h;
  if (i < 0 || i >= m->nt) return -1;
  for (long k = 0; k < m->t[i].numel; ++k) out[k] = to_bf16_bits(m->t[i].v[k]);
  return 0;
}

/* ---- forward helpers working on one activation buffer ---- */

typedef struct {
  double* v;
  int N, H, W, C;
} act_t;

static act_t act_new(int N, int H, int W, int C) {
  act_t a = {malloc(sizeof(double) * (size_t)N * H * W * C), N, H, W, C};
  return a;
}
static long act_numel(const act_t* a) { return (long)a->N * a->H * a->W * a->C; }

static void round_all(double* v, long n, int parity) {
  if (!parity) return;
  for (long i = 0; i < n; ++i) v[i] = oracle_bf16_round(v[i]);
}

/* inference BN with the model's constant statistics: gamma 1, beta 0, mean 0, var 1, eps 1e-5 */
static void bn_const(double* y, long rows, int C) {
  double* one = malloc(sizeof(double) * (size_t)C);
  double* zero = calloc((size_t)C, sizeof(double));
  for (int c = 0; c < C; ++c) one[c] = 1.0;
  batchnorm(y, rows, C, one, zero, zero, one, 1e-5);
  free(one);
  free(zero);
}

enum { ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2 };
static double activate(double v, int act) {
  if (act == ACT_RELU) return v > 0.0 ? v : 0.0;
  if (act == ACT_RELU6) return v < 0.0 ? 0.0 : (v > 6.0 ? 6.0 : v);
  return v;
}

/* conv -> [bias] -> [BN] -> [+ residual] -> act -> (bf16 storage in parity mode) */
static act_t conv_layer(const act_t* x, const double* w, const double* bias, int K, int R, int stride, int pad,
                        int use_bn, const act_t* residual, int act, int parity) {
  act_t y = act_new(x->N, out_dim(x->H, R, stride, pad), out_dim(x->W, R, stride, pad), K);
  oracle_conv2d(x->v, x->N, x->H, x->W, x->C, w, K, R, R, stride, pad, y.v);
  long rows = (long)y.N * y.H * y.W;
  if (bias)
    for (long i = 0; i < rows; ++i)
      for (int k = 0; k < K; ++k) y.v[i * K + k] += bias[k];
  if (use_bn) bn_const(y.v, rows, K);
  for (long i = 0; i < rows * K; ++i) {
    double v = y.v[i] + (residual ? residual->v[i] : 0.0);
    y.v[i] = activate(v, act);
  }
  round_all(y.v, rows * K, parity);
  return y;
}

static act_t dw_layer(const act_t* x, const double* w, int stride, int parity) {
  act_t y = act_new(x->N, out_dim(x->H, 3, stride, 1), out_dim(x->W, 3, stride, 1), x->C);
  oracle_dwconv(x->v, x->N, x->H, x->W, x->C, w, 3, 3, stride, 1, y.v);
  long rows = (long)y.N * y.H * y.W;
  bn_const(y.v, rows, y.C);
  for (long i = 0; i < rows * y.C; ++i) y.v[i] = activate(y.v[i], ACT_RELU6);
  round_all(y.v, rows * y.C, parity);
  return y;
}

static act_t maxpool_layer(const act_t* x, int k, int stride, int pad) {
  act_t y = act_new(x->N, out_dim(x->H, k, stride, pad), out_dim(x->W, k, stride, pad), x->C);
  oracle_maxpool(x->v, x->N, x->H, x->W, x->C, k, stride, pad, y.v);
  return y; /* a max of stored values needs no rounding */
}

static act_t avgpool_layer(const act_t* x, int parity) {
  act_t y = act_new(x->N, 1, 1, x->C);
  oracle_avgpool(x->v, x->N, x->H, x->W, x->C, y.v);
  round_all(y.v, act_numel(&y), parity);
  return y;
}

/* fc on a flattened activation; hidden layers (act != none) are stored as bf16 in parity mode */
static act_t fc_layer(const act_t* x, const double* w, const double* b, int O, int act, int store_bf16,
                      int parity) {
  int I = x->H * x->W * x->C;
  act_t y = act_new(x->N, 1, 1, O);
  oracle_fc(x->v, x->N, I, w, b, O, y.v);
  for (long i = 0; i < act_numel(&y); ++i) y.v[i] = activate(y.v[i], act);
  if (store_bf16) round_all(y.v, act_numel(&y), parity);
  return y;
}

static void act_free(act_t* a) {
  free(a->v);
  a->v = NULL;
}
static void act_replace(act_t* dst, act_t src) {
  act_free(dst);
  *dst = src;
}

static act_t forward_tiny(model_t* m, act_t x, int parity) {
  act_t a = x;
  int ch[5] = {3, 16, 32, 32, 64};
  act_t cur = act_new(a.N, a.H, a.W, a.C);
  memcpy(cur.v, a.v, sizeof(double) * (size_t)act_numel(&a));
  for (int l = 0; l < 4; ++l) {
    act_replace(&cur, conv_layer(&cur, next_tensor(m), NULL, ch[l + 1], 3, 1, 1, 1, NULL, ACT_RELU, parity));
    if (l == 1 || l == 3) act_replace(&cur, maxpool_layer(&cur, 2, 2, 0));
  }
  act_replace(&cur, avgpool_layer(&cur, parity));
  const double* w = next_tensor(m);
  const double* b = next_tensor(m);
  act_replace(&cur, fc_layer(&cur, w, b, 10, ACT_NONE, 0, parity));
  return cur;
}

static act_t forward_r50(model_t* m, act_t x, int parity) {
  act_t cur = conv_layer(&x, next_tensor(m), NULL, 64, 7, 2, 3, 1, NULL, ACT_RELU, parity);
  act_replace(&cur, maxpool_layer(&cur, 3, 2, 1));
  for (int st = 0; st < 4; ++st) {
    int planes = R50_STAGES[st][1];
    for (int b = 0; b < R50_STAGES[st][0]; ++b) {
      int stride = (b == 0) ? R50_STAGES[st][2] : 1;
      const double* w1 = next_tensor(m);
      const double* w2 = next_tensor(m);
      const double* w3 = next_tensor(m);
      act_t t1 = conv_layer(&cur, w1, NULL, planes, 1, 1, 0, 1, NULL, ACT_RELU, parity);
      act_t t2 = conv_layer(&t1, w2, NULL, planes, 3, stride, 1, 1, NULL, ACT_RELU, parity); /* v1.5: stride on 3x3 */
      act_t sc;
      if (b == 0) {
        sc = conv_layer(&cur, next_tensor(m), NULL, 4 * planes, 1, stride, 0, 1, NULL, ACT_NONE, parity);
      } else {
        sc = act_new(cur.N, cur.H, cur.W, cur.C);
        memcpy(sc.v, cur.v, sizeof(double) * (size_t)act_numel(&cur));
      }
      act_t out = conv_layer(&t2, w3, NULL, 4 * planes, 1, 1, 0, 1, &sc, ACT_RELU, parity);
      act_free(&t1);
      act_free(&t2);
      act_free(&sc);
      act_replace(&cur, out);
    }
  }
  act_replace(&cur, avgpool_layer(&cur, parity));
  const double* w = next_tensor(m);
  const double* bb = next_tensor(m);
  act_replace(&cur, fc_layer(&cur, w, bb, 1000, ACT_NONE, 0, parity));
  return cur;
}

static act_t forward_mbv2(model_t* m, act_t x, int parity) {
  act_t cur = conv_layer(&x, next_tensor(m), NULL, 32, 3, 2, 1, 1, NULL, ACT_RELU6, parity);
  int cin = 32;
  for (int g = 0; g < 7; ++g) {
    int t = MBV2_CFG[g][0], c = MBV2_CFG[g][1], n = MBV2_CFG[g][2], s = MBV2_CFG[g][3];
    for (int i = 0; i < n; ++i) {
      int stride = (i == 0) ? s : 1;
      int hid = cin * t;
      act_t e;
      if (t != 1) {
        e = conv_layer(&cur, next_tensor(m), NULL, hid, 1, 1, 0, 1, NULL, ACT_RELU6, parity);
      } else {
        e = act_new(cur.N, cur.H, cur.W, cur.C);
        memcpy(e.v, cur.v, sizeof(double) * (size_t)act_numel(&cur));
      }
      act_t d = dw_layer(&e, next_tensor(m), stride, parity);
      int res = (stride == 1 && cin == c);
      act_t p = conv_layer(&d, next_tensor(m), NULL, c, 1, 1, 0, 1, res ? &cur : NULL, ACT_NONE, parity);
      act_free(&e);
      act_free(&d);
      act_replace(&cur, p);
      cin = c;
    }
  }
  act_replace(&cur, conv_layer(&cur, next_tensor(m), NULL, 1280, 1, 1, 0, 1, NULL, ACT_RELU6, parity));
  act_replace(&cur, avgpool_layer(&cur, parity));
  const double* w = next_tensor(m);
  const double* b = next_tensor(m);
  act_replace(&cur, fc_layer(&cur, w, b, 1000, ACT_NONE, 0, parity));
  return cur;
}

static act_t forward_vgg(model_t* m, act_t x, int parity) {
  act_t cur = act_new(x.N, x.H, x.W, x.C);
  memcpy(cur.v, x.v, sizeof(double) * (size_t)act_numel(&x));
  for (int st = 0; st < 5; ++st) {
    for (int i = 0; i < VGG_STAGE_CONVS[st]; ++i) {
      const double* w = next_tensor(m);
      const double* b = next_tensor(m);
      act_replace(&cur, conv_layer(&cur, w, b, VGG_STAGE_CH[st], 3, 1, 1, 0, NULL, ACT_RELU, parity));
    }
    act_replace(&cur, maxpool_layer(&cur, 2, 2, 0));
  }
  /* flatten in (h, w, c) order: the NHWC buffer already is that order */
  const double *w1 = next_tensor(m), *b1 = next_tensor(m);
  act_replace(&cur, fc_layer(&cur, w1, b1, 4096, ACT_RELU, 1, parity));
  const double *w2 = next_tensor(m), *b2 = next_tensor(m);
  act_replace(&cur, fc_layer(&cur, w2, b2, 4096, ACT_RELU, 1, parity));
  const double *w3 = next_tensor(m), *b3 = next_tensor(m);
  act_replace(&cur, fc_layer(&cur, w3, b3, 1000, ACT_NONE, 0, parity));
  return cur;
}

/* Forward pass of n_items independent samples.
 * CNN: in = [n][H][W][3] bf16 bits, out = [n][classes] fp64.
 * LSTM: in = [50][n][512] bf16 bits, out = [50][n][1024] fp64 (layer-2 h).
 * Returns 0, or -1 for an unknown model or a BERT (oracle_bert_forward). */
int oracle_model_forward(void* h, int n, const uint16_t* in, int parity, double* out) {
  model_t* m = h;
  if (!m || m->arch == ARCH_BERT || m->arch == ARCH_BERT_LONG) return -1; /* token input: oracle_bert_forward */
  m->cursor = 0;
  if (m->arch == ARCH_LSTM) {
    const int T = 50, I = 512, Hd = 1024;
    double* x = malloc(sizeof(double) * (size_t)T * n * I);
    for (long i = 0; i < (long)T * n * I; ++i) x[i] = oracle_bf16_to_double(in[i]);
    double* h1 = malloc(sizeof(double) * (size_t)T * n * Hd);
    const double *wi0 = next_tensor(m), *wh0 = next_tensor(m), *bi0 = next_tensor(m), *bh0 = next_tensor(m);
    oracle_lstm_layer(x, T, n, I, Hd, wi0, wh0, bi0, bh0, parity, h1, NULL);
    round_all(h1, (long)T * n * Hd, parity); /* layer-2 input enters a product */
    const double *wi1 = next_tensor(m), *wh1 = next_tensor(m), *bi1 = next_tensor(m), *bh1 = next_tensor(m);
    oracle_lstm_layer(h1, T, n, Hd, Hd, wi1, wh1, bi1, bh1, parity, out, NULL);
    free(x);
    free(h1);
    return 0;
  }
  int HW = (m->arch == ARCH_TINY) ? 32 : 224;
  act_t x = act_new(n, HW, HW, 3);
  for (long i = 0; i < act_numel(&x); ++i) x.v[i] = oracle_bf16_to_double(in[i]);
  act_t y;
  switch (m->arch) {
    case ARCH_TINY: y = forward_tiny(m, x, parity); break;
    case ARCH_R50: y = forward_r50(m, x, parity); break;
    case ARCH_MBV2: y = forward_mbv2(m, x, parity); break;
    default: y = forward_vgg(m, x, parity); break;
  }
  memcpy(out, y.v, sizeof(double) * (size_t)act_numel(&y));
  act_free(&x);
  act_free(&y);
  return 0;
}

/* ---- BERT encoder ---- */

static double gelu(double v) { return 0.5 * v * (1.0 + erf(v / sqrt(2.0))); }

/* y [rows][O] = x [rows][I] w^T + b (+ res) then act (0 none, 3 GELU, 4
 * tanh), bf16 storage in parity mode */
static void bert_linear(const double* x, long rows, int I, const double* w, const double* b, int O,
                        const double* res, int act, int parity, double* y) {
  oracle_fc(x, (int)rows, I, w, b, O, y);
  for (long i = 0; i < rows * O; ++i) {
    double v = y[i] + (res ? res[i] : 0.0);
    if (act == 3) v = gelu(v);
    if (act == 4) v = tanh(v);
    y[i] = v;
  }
  round_all(y, rows * O, parity);
}

static void bert_ln(double* x, long rows, int parity) {
  double* g = malloc(sizeof(double) * BERT_H);
  double* z = calloc(BERT_H, sizeof(double));
  for (int c = 0; c < BERT_H; ++c) g[c] = 1.0;
  oracle_layernorm(x, rows, BERT_H, g, z, 1e-12, x);
  round_all(x, rows * BERT_H, parity);
  free(g);
  free(z);
}

/* Forward pass of n sequences of T token ids (token type 0, no padding):
 * embeddings (word + position + type) -> layer norm -> 12 post-norm encoder
 * layers (self-attention + residual -> layer norm, GELU feed-forward +
 * residual -> layer norm) -> pooler tanh(W_p h_[CLS] + b_p) -> classifier,
 * out [n][2] fp64.  T is 20 for "bert" and 40 for "bert_long".  Returns 0,
 * or -1 for a model that is not a BERT or an id outside the vocabulary. */
/* Encoder layer l (1..12) of n sequences of T tokens, in place on x
 * [n*T][768]: self-attention + residual -> layer norm, GELU feed-forward +
 * residual -> layer norm (bf16 storage after each step in parity mode).
 * Its tensors are 3 + 8 (l - 1) .. + 7 (after the three embedding tables). */
static void bert_layer(model_t* m, int l, int n, int T, int parity, double* x) {
  const long rows = (long)n * T;
  const tensor_t* t = &m->t[3 + 8 * (l - 1)];
  const double *wqkv = t[0].v, *bqkv = t[1].v, *wo = t[2].v, *bo = t[3].v;
  const double *w1 = t[4].v, *b1 = t[5].v, *w2 = t[6].v, *b2 = t[7].v;
  double* qkv = malloc(sizeof(double) * (size_t)rows * 3 * BERT_H);
  double* att = malloc(sizeof(double) * (size_t)rows * BERT_H);
  double* a = malloc(sizeof(double) * (size_t)rows * BERT_H);
  double* f = malloc(sizeof(double) * (size_t)rows * BERT_FF);
  bert_linear(x, rows, BERT_H, wqkv, bqkv, 3 * BERT_H, NULL, 0, parity, qkv);
  oracle_attention(qkv, n, T, BERT_HEADS, BERT_DH, att);
  round_all(att, rows * BERT_H, parity);
  bert_linear(att, rows, BERT_H, wo, bo, BERT_H, x, 0, parity, a);
  bert_ln(a, rows, parity);
  bert_linear(a, rows, BERT_H, w1, b1, BERT_FF, NULL, 3, parity, f);
  bert_linear(f, rows, BERT_FF, w2, b2, BERT_H, a, 0, parity, x);
  bert_ln(x, rows, parity);
  free(qkv);
  free(att);
  free(a);
  free(f);
}

/* The encoder up to layer `layers` (0: the embeddings word + position +
 * type and their layer norm): x [n*T][768] receives that hidden state. */
static void bert_encode(model_t* m, int n, int T, const int32_t* ids, int parity, int layers, double* x) {
  const long rows = (long)n * T;
  const double *we = m->t[0].v, *pe = m->t[1].v, *te = m->t[2].v;
  for (long r = 0; r < rows; ++r) {
    const int t = (int)(r % T);
    for (int c = 0; c < BERT_H; ++c)
      x[r * BERT_H + c] = we[(long)ids[r] * BERT_H + c] + pe[(long)t * BERT_H + c] + te[c];
  }
  bert_ln(x, rows, parity);
  for (int l = 1; l <= layers; ++l) bert_layer(m, l, n, T, parity, x);
}

static int bert_check(model_t* m, int n, const int32_t* ids) {
  if (!m || (m->arch != ARCH_BERT && m->arch != ARCH_BERT_LONG)) return -1;
  const long rows = (long)n * (m->arch == ARCH_BERT ? 20 : 40);
  for (long i = 0; i < rows; ++i)
    if (ids[i] < 0 || ids[i] >= BERT_VOCAB) return -1;
  return 0;
}

/* The hidden state [n][T][768] after encoder layer `layers` (0: the
 * embeddings; 12: the encoder's output), a test hook beside the classifier
 * output of oracle_bert_forward.  Returns 0, or -1 as it (or a layer
 * outside 0..12). */
int oracle_bert_hidden(void* h, int n, const int32_t* ids, int parity, int layers, double* out) {
  model_t* m = h;
  if (bert_check(m, n, ids) || layers < 0 || layers > BERT_L) return -1;
  bert_encode(m, n, m->arch == ARCH_BERT ? 20 : 40, ids, parity, layers, out);
  return 0;
}

/* Encoder layer l (1..12) alone on a given input x_in [n][T][768] (its
 * values used as they are), into x_out: per-layer parity with the GPU's own
 * bf16 layer input.  Returns 0 or -1. */
int oracle_bert_layer(void* h, int n, int l, const double* x_in, int parity, double* x_out) {
  model_t* m = h;
  if (!m || (m->arch != ARCH_BERT && m->arch != ARCH_BERT_LONG) || l < 1 || l > BERT_L) return -1;
  const int T = m->arch == ARCH_BERT ? 20 : 40;
  memcpy(x_out, x_in, sizeof(double) * (size_t)n * T * BERT_H);
  bert_layer(m, l, n, T, parity, x_out);
  return 0;
}

int oracle_bert_forward(void* h, int n, const int32_t* ids, int parity, double* out) {
  model_t* m = h;
  if (bert_check(m, n, ids)) return -1;
  const int T = m->arch == ARCH_BERT ? 20 : 40;
  double* x = malloc(sizeof(double) * (size_t)n * T * BERT_H);
  bert_encode(m, n, T, ids, parity, BERT_L, x);
  m->cursor = 3 + 8 * BERT_L;
  const double *wp = next_tensor(m), *bp = next_tensor(m), *wc = next_tensor(m), *bc = next_tensor(m);
  double* cls = malloc(sizeof(double) * (size_t)n * BERT_H);
  double* pooled = malloc(sizeof(double) * (size_t)n * BERT_H);
  for (int b = 0; b < n; ++b) memcpy(cls + (long)b * BERT_H, x + (long)b * T * BERT_H, sizeof(double) * BERT_H);
  bert_linear(cls, n, BERT_H, wp, bp, BERT_H, NULL, 4, parity, pooled);
  oracle_fc(pooled, n, BERT_H, wc, bc, BERT_CLASSES, out);
  free(x);
  free(cls);
  free(pooled);
  return 0;
}
