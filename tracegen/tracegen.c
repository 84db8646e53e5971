/*
 * tracegen.c -- seeded synthetic allocate/free traces shaped like the training
 * workloads the paper profiles (Table 2: CNNs and Transformers; three or more
 * iterations with zero_grad, forward, backward, optimizer step; Section 3.3's
 * lifetime rules for parameters, batch data, activations, gradients and
 * optimizer state).  The paper's own profiler traces are not available, so
 * these stand in for them.
 *
 * This module only writes event words (bit 63 = free, low 32 bits = index of
 * the freed allocation; otherwise the requested byte count).  It contains no
 * allocator logic: no rounding, pools, segments or fits.
 *
 * Random numbers: SplitMix64 (Steele, Lea, Flood 2014) seeds xoshiro256**
 * (Blackman, Vigna 2018); each trace has its own stream seeded from
 * (config << 32 | trace_index) ^ seed.
 *
 * Configurations (all sizes in bytes):
 *   1  MLP, 12 layers, 3 iterations, strictly LIFO, balanced, sizes
 *      log-uniform in [1 KiB, 8 MiB] rounded to 4 B, drawn once per
 *      (layer, role); padded with nested temporaries to the exact length.
 *   2  ResNet-50-like CNN, fp32, 224x224 input, batch 16 + floor(496 t / 255);
 *      a workspace temporary uniform in [0, 64 MiB] (4 B steps) around every
 *      convolution in forward and backward; zero_grad frees gradients at the
 *      start of each iteration; SGD without state.
 *   3  GPT-style decoder, 24 layers, hidden {1024,2048,4096}[t%3],
 *      seq {512,1024,2048}[(t/3)%3], batch 1 + (t/9)%16, vocab 50304;
 *      bf16 activations, fp32 parameters and gradients, Adam moments (2x
 *      parameters, fp32) allocated at the first step and kept; flash-style
 *      attention saves only a [b, heads, s] fp32 log-sum-exp; after every op a
 *      temporary with probability 1/2, log-uniform in [512, op output], freed
 *      1-4 events later.
 *   4  Monte Carlo perturbation of 3: base shape t % 144, own seed, every
 *      nonzero size jittered by floor(s * j / 100000), j uniform in
 *      [-10000, 10000], rounded up to 4 B (min 4); each maximal run of
 *      consecutive frees is cut into chunks of 8 that are shuffled
 *      (Fisher-Yates), which keeps every free after its allocation.
 *   5  config 3 at hidden 2048, seq 1024, batch 8, plus one fragmentation
 *      phase after the first iteration: 2 * frag_pairs temporaries of
 *      512 B .. 64 KiB (512 B steps), every other one freed at once, the rest
 *      kept for the whole trace.
 * Every trace stops at exactly the requested number of events; allocations
 * still live then stay live (persistent), except config 1, which is balanced.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define FREE_BIT (1ull << 63)

/* ---------------- random numbers ---------------- */
typedef struct { uint64_t s[4]; } rng_t;

static uint64_t splitmix64(uint64_t* x) {
  uint64_t z = (*x += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
static uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }
static uint64_t next64(rng_t* r) {
  uint64_t* s = r->s;
  const uint64_t result = rotl(s[1] * 5, 7) * 9;
  const uint64_t t = s[1] << 17;
  s[2] ^= s[0]; s[3] ^= s[1]; s[1] ^= s[2]; s[0] ^= s[3];
  s[2] ^= t;
  s[3] = rotl(s[3], 45);
  return result;
}
static void rng_seed(rng_t* r, uint64_t seed) {
  uint64_t x = seed;
  for (int i = 0; i < 4; ++i) r->s[i] = splitmix64(&x);
}
static double unif(rng_t* r) { return (double)(next64(r) >> 11) * (1.0 / 9007199254740992.0); }
/* uniform integer in [0, n) */
static uint64_t below(rng_t* r, uint64_t n) { return (uint64_t)(((__uint128_t)next64(r) * n) >> 64); }
static uint64_t round4(double x) {
  uint64_t v = (uint64_t)x;
  return (v + 3) & ~3ull;
}
/* log-uniform in [lo, hi], rounded up to 4 B */
static uint64_t loguni(rng_t* r, double lo, double hi) {
  if (hi <= lo) return round4(lo);
  return round4(exp(log(lo) + unif(r) * (log(hi) - log(lo))));
}

/* ---------------- trace builder ---------------- */
#define MAX_PENDING 64
typedef struct {
  uint64_t* ev;
  int64_t n, cap;
  rng_t rng;
  /* short-lived temporaries: handle and events left before the free */
  int64_t pend_h[MAX_PENDING];
  int pend_k[MAX_PENDING];
  int npend;
} tb_t;

static int full(const tb_t* b) { return b->n >= b->cap; }

static int64_t emit_alloc(tb_t* b, uint64_t bytes) {
  if (full(b)) return -1;
  b->ev[b->n] = bytes & ~FREE_BIT;
  return b->n++;
}
static void emit_free(tb_t* b, int64_t h) {
  if (h < 0 || full(b)) return;
  b->ev[b->n++] = FREE_BIT | (uint64_t)h;
}
/* one event has passed: release temporaries whose time is up */
static void tick(tb_t* b) {
  int w = 0;
  for (int i = 0; i < b->npend; ++i) {
    if (--b->pend_k[i] <= 0) emit_free(b, b->pend_h[i]);
    else { b->pend_h[w] = b->pend_h[i]; b->pend_k[w] = b->pend_k[i]; ++w; }
  }
  b->npend = w;
}
static int64_t talloc(tb_t* b, uint64_t bytes) { int64_t h = emit_alloc(b, bytes); tick(b); return h; }
static void tfree(tb_t* b, int64_t h) { if (h >= 0 && !full(b)) { emit_free(b, h); tick(b); } }
/* with probability 1/2, a temporary log-uniform in [512, out_bytes], freed 1-4 events later */
static void maybe_temp(tb_t* b, uint64_t out_bytes) {
  if (next64(&b->rng) >> 63) return;
  uint64_t sz = loguni(&b->rng, 512.0, (double)(out_bytes > 512 ? out_bytes : 512));
  int k = 1 + (int)below(&b->rng, 4);
  int64_t h = emit_alloc(b, sz);
  if (h >= 0 && b->npend < MAX_PENDING) { b->pend_h[b->npend] = h; b->pend_k[b->npend] = k; b->npend++; }
  else if (h >= 0) emit_free(b, h);
  tick(b);
}

/* ---------------- config 1: LIFO MLP ---------------- */
static int gen_mlp(tb_t* b) {
  enum { L = 12, ITERS = 3, K = 27 };
  /* 24 params + per iteration 12 * (2 + 4K) + 24 param frees */
  const int64_t base = 2 * 2 * L + (int64_t)ITERS * L * (2 + 4 * K);
  const int64_t pad = b->cap - base;
  if (pad < 0 || (pad & 1)) return -1;
  uint64_t w[L], bi[L], act[L], tf[L][K], tbk[L][K];
  for (int l = 0; l < L; ++l) {
    w[l] = loguni(&b->rng, 1024, 8 << 20);
    bi[l] = loguni(&b->rng, 1024, 8 << 20);
    act[l] = loguni(&b->rng, 1024, 8 << 20);
    for (int j = 0; j < K; ++j) { tf[l][j] = loguni(&b->rng, 1024, 8 << 20); tbk[l][j] = loguni(&b->rng, 1024, 8 << 20); }
  }
  int64_t pw[L], pb[L], ha[L];
  for (int l = 0; l < L; ++l) { pw[l] = emit_alloc(b, w[l]); pb[l] = emit_alloc(b, bi[l]); }
  for (int it = 0; it < ITERS; ++it) {
    for (int l = 0; l < L; ++l) {
      ha[l] = emit_alloc(b, act[l]);
      for (int j = 0; j < K; ++j) emit_free(b, emit_alloc(b, tf[l][j]));
    }
    for (int l = L - 1; l >= 0; --l) {
      for (int j = 0; j < K; ++j) emit_free(b, emit_alloc(b, tbk[l][j]));
      if (it == ITERS - 1 && l == 0)
        for (int64_t j = 0; j < pad / 2; ++j) emit_free(b, emit_alloc(b, tbk[(j / K) % L][j % K]));
      emit_free(b, ha[l]);
    }
  }
  for (int l = L - 1; l >= 0; --l) { emit_free(b, pb[l]); emit_free(b, pw[l]); }
  return b->n == b->cap ? 0 : -1;
}

/* ---------------- config 2: ResNet-50-like CNN ---------------- */
enum { OP_CONV, OP_BN, OP_RELU, OP_MAXPOOL, OP_ADD, OP_AVGPOOL, OP_FC };
typedef struct {
  int kind;
  uint64_t in_b, out_b, w_b;  /* per-sample input / output bytes; weight bytes */
  int c;                      /* channels (BN) */
} cnn_op;

static int build_resnet50(cnn_op* ops) {
  int n = 0;
  const uint64_t F4 = 4;
#define PUSH(k, ib, ob, wb, cc) do { ops[n].kind = (k); ops[n].in_b = (ib); ops[n].out_b = (ob); ops[n].w_b = (wb); ops[n].c = (cc); ++n; } while (0)
  uint64_t a = 3ull * 224 * 224 * F4;
  uint64_t o = 64ull * 112 * 112 * F4;
  PUSH(OP_CONV, a, o, 64ull * 3 * 49 * F4, 64);
  PUSH(OP_BN, o, o, 0, 64);
  PUSH(OP_RELU, o, o, 0, 0);
  a = o; o = 64ull * 56 * 56 * F4;
  PUSH(OP_MAXPOOL, a, o, 0, 0);
  const int blocks[4] = {3, 4, 6, 3}, mid[4] = {64, 128, 256, 512}, outc[4] = {256, 512, 1024, 2048},
            hw[4] = {56, 28, 14, 7};
  int cin = 64, hin = 56;
  for (int s = 0; s < 4; ++s)
    for (int k = 0; k < blocks[s]; ++k) {
      const uint64_t x = (uint64_t)cin * hin * hin * F4;
      const uint64_t m1 = (uint64_t)mid[s] * hin * hin * F4;
      const uint64_t m2 = (uint64_t)mid[s] * hw[s] * hw[s] * F4;
      const uint64_t y = (uint64_t)outc[s] * hw[s] * hw[s] * F4;
      PUSH(OP_CONV, x, m1, (uint64_t)mid[s] * cin * F4, mid[s]);
      PUSH(OP_BN, m1, m1, 0, mid[s]);
      PUSH(OP_RELU, m1, m1, 0, 0);
      PUSH(OP_CONV, m1, m2, (uint64_t)mid[s] * mid[s] * 9 * F4, mid[s]);
      PUSH(OP_BN, m2, m2, 0, mid[s]);
      PUSH(OP_RELU, m2, m2, 0, 0);
      PUSH(OP_CONV, m2, y, (uint64_t)outc[s] * mid[s] * F4, outc[s]);
      PUSH(OP_BN, y, y, 0, outc[s]);
      if (k == 0) {
        PUSH(OP_CONV, x, y, (uint64_t)outc[s] * cin * F4, outc[s]);
        PUSH(OP_BN, y, y, 0, outc[s]);
      }
      PUSH(OP_ADD, y, y, 0, 0);
      PUSH(OP_RELU, y, y, 0, 0);
      cin = outc[s];
      hin = hw[s];
    }
  PUSH(OP_AVGPOOL, 2048ull * 49 * F4, 2048ull * F4, 0, 0);
  PUSH(OP_FC, 2048ull * F4, 1000ull * F4, 2048ull * 1000 * F4, 1000);
#undef PUSH
  return n;
}

static uint64_t ws_size(tb_t* b) { return below(&b->rng, (64ull << 20) / 4 + 1) * 4; }

#define MAX_OPS 256
static int gen_cnn(tb_t* b, uint64_t batch) {
  cnn_op ops[MAX_OPS];
  const int n = build_resnet50(ops);
  /* parameters: conv weight; BN weight, bias, running mean, running var; fc weight, bias */
  for (int i = 0; i < n; ++i) {
    if (ops[i].kind == OP_CONV) emit_alloc(b, ops[i].w_b);
    if (ops[i].kind == OP_BN) for (int j = 0; j < 4; ++j) emit_alloc(b, (uint64_t)ops[i].c * 4);
    if (ops[i].kind == OP_FC) { emit_alloc(b, ops[i].w_b); emit_alloc(b, (uint64_t)ops[i].c * 4); }
  }
  static __thread int64_t grads[4 * MAX_OPS];
  int ngrad = 0;
  int64_t saved[MAX_OPS][3];
  while (!full(b)) {
    for (int g = 0; g < ngrad; ++g) emit_free(b, grads[g]);  /* zero_grad(set_to_none) */
    ngrad = 0;
    const int64_t x = emit_alloc(b, batch * 3 * 224 * 224 * 4);
    const int64_t y = emit_alloc(b, batch * 8);
    for (int i = 0; i < n; ++i) {
      const cnn_op* o = &ops[i];
      saved[i][0] = saved[i][1] = saved[i][2] = -1;
      switch (o->kind) {
        case OP_CONV: {
          const int64_t ws = emit_alloc(b, ws_size(b));
          saved[i][0] = emit_alloc(b, batch * o->out_b);
          emit_free(b, ws);
        } break;
        case OP_BN:
          saved[i][0] = emit_alloc(b, batch * o->out_b);
          saved[i][1] = emit_alloc(b, (uint64_t)o->c * 4);
          saved[i][2] = emit_alloc(b, (uint64_t)o->c * 4);
          break;
        case OP_MAXPOOL:
          saved[i][0] = emit_alloc(b, batch * o->out_b);
          saved[i][1] = emit_alloc(b, batch * o->out_b * 2);
          break;
        case OP_ADD: case OP_AVGPOOL: case OP_FC:
          saved[i][0] = emit_alloc(b, batch * o->out_b);
          break;
        default: break;  /* ReLU in place */
      }
    }
    const int64_t sm = emit_alloc(b, batch * 1000 * 4);
    const int64_t loss = emit_alloc(b, 4);
    int64_t gout = emit_alloc(b, batch * 1000 * 4);
    emit_free(b, loss);
    emit_free(b, sm);
    for (int i = n - 1; i >= 0; --i) {
      const cnn_op* o = &ops[i];
      int64_t gin = -1;
      switch (o->kind) {
        case OP_CONV: {
          int64_t ws = emit_alloc(b, ws_size(b));
          if (i > 0) gin = emit_alloc(b, batch * o->in_b);
          emit_free(b, ws);
          ws = emit_alloc(b, ws_size(b));
          grads[ngrad++] = emit_alloc(b, o->w_b);
          emit_free(b, ws);
        } break;
        case OP_BN:
          gin = emit_alloc(b, batch * o->in_b);
          grads[ngrad++] = emit_alloc(b, (uint64_t)o->c * 4);
          grads[ngrad++] = emit_alloc(b, (uint64_t)o->c * 4);
          break;
        case OP_FC:
          gin = emit_alloc(b, batch * o->in_b);
          grads[ngrad++] = emit_alloc(b, o->w_b);
          grads[ngrad++] = emit_alloc(b, (uint64_t)o->c * 4);
          break;
        case OP_ADD:
          gin = emit_alloc(b, batch * o->in_b);  /* gradient of the shortcut sum */
          break;
        default:
          gin = emit_alloc(b, batch * o->in_b);
          break;
      }
      if (gin >= 0 || i == 0) {
        emit_free(b, gout);
        gout = gin;
      }
      for (int j = 2; j >= 0; --j) emit_free(b, saved[i][j]);
    }
    emit_free(b, gout);
    emit_free(b, y);
    emit_free(b, x);
  }
  return 0;
}

/* ---------------- config 3/4/5: GPT-style decoder ---------------- */
typedef struct { uint64_t h, s, bt, V; int L; } gpt_shape;

static gpt_shape gpt_shape_of(int64_t t) {
  static const uint64_t H[3] = {1024, 2048, 4096}, S[3] = {512, 1024, 2048};
  gpt_shape g = {H[t % 3], S[(t / 3) % 3], 1 + (uint64_t)((t / 9) % 16), 50304, 24};
  return g;
}

/* per layer parameter sizes (fp32): ln1 w,b; qkv w,b; proj w,b; ln2 w,b; fc1 w,b; fc2 w,b */
static void layer_params(uint64_t h, uint64_t* p) {
  const uint64_t v[12] = {h, h, h * 3 * h, 3 * h, h * h, h, h, h, h * 4 * h, 4 * h, 4 * h * h, h};
  for (int i = 0; i < 12; ++i) p[i] = v[i] * 4;
}

static void frag_phase(tb_t* b, int64_t pairs) {
  for (int64_t i = 0; i < pairs && !full(b); ++i) {
    const int64_t keep = emit_alloc(b, 512 * (1 + below(&b->rng, 128)));
    const int64_t drop = emit_alloc(b, 512 * (1 + below(&b->rng, 128)));
    (void)keep;
    (void)drop;
  }
  /* free every other one of the block just emitted: the second of each pair */
  const int64_t end = b->n;
  const int64_t start = end - 2 * pairs;
  for (int64_t k = start + 1; k < end && !full(b); k += 2) emit_free(b, k);
}

static int gen_gpt(tb_t* b, gpt_shape g, int64_t frag_pairs) {
  const uint64_t h = g.h, s = g.s, bt = g.bt, V = g.V;
  const uint64_t heads = h / 64;
  const uint64_t bs = bt * s, act = bs * h * 2, act3 = bs * 3 * h * 2, act4 = bs * 4 * h * 2;
  const int L = g.L;
  uint64_t lp[12];
  layer_params(h, lp);
  /* model.to(device): persistent parameters */
  const uint64_t other_p[4] = {V * h * 4, s * h * 4, h * 4, h * 4};  /* wte, wpe, ln_f w, b */
  for (int l = 0; l < L; ++l) for (int i = 0; i < 12; ++i) emit_alloc(b, lp[i]);
  for (int i = 0; i < 4; ++i) emit_alloc(b, other_p[i]);
  static __thread int64_t grads[24 * 12 + 8];
  int ngrad = 0, iter = 0;
  /* per layer saved tensors: ln1 out/mean/rstd, qkv, attn out, lse, proj, add1, ln2 out/mean/rstd, fc1, gelu, fc2, add2 */
  int64_t sv[24][16];
  while (!full(b)) {
    for (int i = 0; i < ngrad; ++i) tfree(b, grads[i]);  /* zero_grad at iteration start */
    ngrad = 0;
    const int64_t tok = talloc(b, bs * 8), tgt = talloc(b, bs * 8);
    const int64_t emb = talloc(b, act);
    maybe_temp(b, act);
    for (int l = 0; l < L; ++l) {
      int64_t* v = sv[l];
      v[0] = talloc(b, act); v[1] = talloc(b, bs * 4); v[2] = talloc(b, bs * 4); maybe_temp(b, act);
      v[3] = talloc(b, act3); maybe_temp(b, act3);
      v[4] = talloc(b, act); v[5] = talloc(b, bt * heads * s * 4); maybe_temp(b, act);
      v[6] = talloc(b, act); maybe_temp(b, act);
      v[7] = talloc(b, act); maybe_temp(b, act);
      v[8] = talloc(b, act); v[9] = talloc(b, bs * 4); v[10] = talloc(b, bs * 4); maybe_temp(b, act);
      v[11] = talloc(b, act4); maybe_temp(b, act4);
      v[12] = talloc(b, act4); maybe_temp(b, act4);
      v[13] = talloc(b, act); maybe_temp(b, act);
      v[14] = talloc(b, act); maybe_temp(b, act);
    }
    const int64_t lnf = talloc(b, act), lnf_m = talloc(b, bs * 4), lnf_r = talloc(b, bs * 4);
    maybe_temp(b, act);
    const int64_t logits = talloc(b, bs * V * 2);
    maybe_temp(b, bs * V * 2);
    const int64_t lsm = talloc(b, bs * V * 4);  /* fp32 log-softmax, saved for backward */
    const int64_t loss = talloc(b, 4);
    /* backward */
    int64_t g = talloc(b, bs * V * 2);
    tfree(b, loss);
    tfree(b, lsm);
    maybe_temp(b, bs * V * 2);
    int64_t gi = talloc(b, act);
    grads[ngrad++] = talloc(b, V * h * 4); /* tied embedding gradient */
    tfree(b, g); tfree(b, logits); g = gi;
    maybe_temp(b, act);
    gi = talloc(b, act); grads[ngrad++] = talloc(b, h * 4); grads[ngrad++] = talloc(b, h * 4);
    tfree(b, g); tfree(b, lnf); tfree(b, lnf_m); tfree(b, lnf_r); g = gi;
    for (int l = L - 1; l >= 0; --l) {
      int64_t* v = sv[l];
      /* fc2: grad in (4h), weight and bias grads */
      gi = talloc(b, act4); grads[ngrad++] = talloc(b, lp[10]); grads[ngrad++] = talloc(b, lp[11]);
      tfree(b, g); tfree(b, v[14]); tfree(b, v[13]); g = gi; maybe_temp(b, act4);
      gi = talloc(b, act4); tfree(b, g); tfree(b, v[12]); g = gi; maybe_temp(b, act4);   /* gelu */
      gi = talloc(b, act); grads[ngrad++] = talloc(b, lp[8]); grads[ngrad++] = talloc(b, lp[9]);
      tfree(b, g); tfree(b, v[11]); g = gi; maybe_temp(b, act);                          /* fc1 */
      gi = talloc(b, act); grads[ngrad++] = talloc(b, lp[6]); grads[ngrad++] = talloc(b, lp[7]);
      tfree(b, g); tfree(b, v[8]); tfree(b, v[9]); tfree(b, v[10]); g = gi; maybe_temp(b, act);  /* ln2 */
      gi = talloc(b, act); tfree(b, g); tfree(b, v[7]); g = gi;                         /* residual */
      gi = talloc(b, act); grads[ngrad++] = talloc(b, lp[4]); grads[ngrad++] = talloc(b, lp[5]);
      tfree(b, g); tfree(b, v[6]); g = gi; maybe_temp(b, act);                           /* proj */
      gi = talloc(b, act3); tfree(b, g); tfree(b, v[4]); tfree(b, v[5]); g = gi; maybe_temp(b, act3); /* attn */
      gi = talloc(b, act); grads[ngrad++] = talloc(b, lp[2]); grads[ngrad++] = talloc(b, lp[3]);
      tfree(b, g); tfree(b, v[3]); g = gi; maybe_temp(b, act);                           /* qkv */
      gi = talloc(b, act); grads[ngrad++] = talloc(b, lp[0]); grads[ngrad++] = talloc(b, lp[1]);
      tfree(b, g); tfree(b, v[0]); tfree(b, v[1]); tfree(b, v[2]); g = gi; maybe_temp(b, act);  /* ln1 */
    }
    grads[ngrad++] = talloc(b, s * h * 4);  /* position embedding gradient */
    tfree(b, g); tfree(b, emb);
    if (iter == 0) {  /* Adam: exp_avg and exp_avg_sq for every parameter, kept */
      for (int l = 0; l < L; ++l) for (int i = 0; i < 12; ++i) { talloc(b, lp[i]); talloc(b, lp[i]); }
      for (int i = 0; i < 4; ++i) { talloc(b, other_p[i]); talloc(b, other_p[i]); }
    }
    tfree(b, tgt); tfree(b, tok);
    if (iter == 0 && frag_pairs > 0) frag_phase(b, frag_pairs);
    ++iter;
  }
  return 0;
}

/* ---------------- config 4 post-processing ---------------- */
static void jitter_sizes(tb_t* b) {
  for (int64_t i = 0; i < b->n; ++i) {
    uint64_t w = b->ev[i];
    if (w & FREE_BIT || w == 0) continue;
    const int64_t j = (int64_t)below(&b->rng, 20001) - 10000;
    int64_t s = (int64_t)w;
    const __int128 d = (__int128)s * j;
    s += (int64_t)(d >= 0 ? d / 100000 : -((-d + 99999) / 100000));  /* floor division */
    uint64_t r = ((uint64_t)s + 3) & ~3ull;
    b->ev[i] = r < 4 ? 4 : r;
  }
}

static void shuffle_free_runs(tb_t* b) {
  int64_t i = 0;
  while (i < b->n) {
    if (!(b->ev[i] & FREE_BIT)) { ++i; continue; }
    int64_t j = i;
    while (j < b->n && (b->ev[j] & FREE_BIT)) ++j;
    for (int64_t c = i; c < j; c += 8) {
      const int64_t m = (j - c) < 8 ? (j - c) : 8;
      for (int64_t k = m - 1; k > 0; --k) {
        const int64_t r = (int64_t)below(&b->rng, (uint64_t)k + 1);
        const uint64_t t = b->ev[c + k]; b->ev[c + k] = b->ev[c + r]; b->ev[c + r] = t;
      }
    }
    i = j;
  }
}

/* ---------------- public entry points ---------------- */
int64_t tg_default_traces(int config) {
  switch (config) { case 1: return 1; case 2: return 256; case 3: return 1024; case 4: return 4096; case 5: return 1; }
  return -1;
}
int64_t tg_default_events(int config) {
  switch (config) { case 1: return 4096; case 2: return 65536; case 3: return 262144; case 4: return 65536; case 5: return 16777216; }
  return -1;
}

/* Fill out[0..n_events) with trace `trace_index` of `config`.  frag_pairs is
 * used by config 5 only (< 0 selects the default).  Returns 0, or -1 if the
 * configuration or length is not supported. */
int tg_trace(int config, int64_t trace_index, uint64_t seed, int64_t frag_pairs, uint64_t* out, int64_t n_events);

/* As tg_trace, stopping config 4's post-processing early: stage 0 is the base
 * trace (before the size jitter), 1 the jittered one (before the free-run
 * shuffle), 2 the final trace.  Other configurations ignore the stage. */
int tg_trace_stage(int config, int64_t trace_index, uint64_t seed, int64_t frag_pairs, uint64_t* out, int64_t n_events,
                   int stage) {
  if (n_events < 0 || (n_events > 0 && !out)) return -1;
  tb_t b;
  memset(&b, 0, sizeof b);
  b.ev = out;
  b.cap = n_events;
  rng_seed(&b.rng, (((uint64_t)config << 32) | (uint64_t)trace_index) ^ seed);
  switch (config) {
    case 1: return gen_mlp(&b);
    case 2: return gen_cnn(&b, 16 + (uint64_t)(496 * trace_index / 255));
    case 3: return gen_gpt(&b, gpt_shape_of(trace_index), 0);
    case 4: {
      int rc = gen_gpt(&b, gpt_shape_of(trace_index % 144), 0);
      if (stage >= 1) jitter_sizes(&b);
      if (stage >= 2) shuffle_free_runs(&b);
      return rc;
    }
    case 5: {
      gpt_shape g = {2048, 1024, 8, 50304, 24};
      return gen_gpt(&b, g, frag_pairs < 0 ? 67000 : frag_pairs);
    }
  }
  return -1;
}

int tg_trace(int config, int64_t trace_index, uint64_t seed, int64_t frag_pairs, uint64_t* out, int64_t n_events) {
  return tg_trace_stage(config, trace_index, seed, frag_pairs, out, n_events, 2);
}
