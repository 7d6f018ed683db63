/*
 * tempo_oracle.c -- plain, slow, obviously-correct CPU oracle for one GPU's
 * share of the expert-parallel MoE block (TEMPO: makespan-aware
 * expert-parallel load balancing).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may link, load or
 * call this file; only the test-suite, the smoke check and the CPU-baseline
 * leg of the benchmark do.  It shares no code, header, table or constant
 * generator with the HIP library.
 *
 * What it computes (paper passages in brackets):
 *   oracle_dispatch  -- stage 1: per-expert histogram of the routed
 *                       (token, k) pairs, per-replica split of each expert's
 *                       tokens following the per-batch plan, padding of every
 *                       local replica slot to whole M-tiles, and the stable
 *                       permutation of pairs into those padded groups.
 *                       [Sec. 3.1 fixed-charge problem: n_e, R(e), x_{e,g},
 *                        z_{e,g}; Sec. 2.2 / Eq. 2: M-tiles, T = sum ceil(n/128);
 *                        Sec. 4.4 integration: counts masked against graph
 *                        padding rows, cumulative counter, rows renormalised
 *                        at use, zero-sum row -> uniform over replicas.]
 *   oracle_moe       -- stages 2+3: per local pair, gate/up projection,
 *                       SwiGLU, down projection, then the routing-weighted
 *                       sum over k.  [Sec. 2.1: grouped expert GEMMs
 *                       "gate/up, activation, down" followed by combine.]
 *
 * Everything is double precision except where an exact integer is defined.
 * Two modes for stage 2/3:
 *   mode 0 (exact)  -- h, o and y are never rounded.
 *   mode 1 (mirror) -- rounds h (bf16, or fp8 e4m3 with 1x128 block scales),
 *                      o and y (bf16) at the points a bf16/fp8 datapath
 *                      stores them; the dot products stay in fp64.
 *
 * Parity pins live in tests/ (brute force, invariants, special cases that
 * reduce to library routines, the dense-FFN reduction, split invariance).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* sticky data-error bits, one per class of bad input */
#define ORC_ERR_BAD_ID 1u          /* routing id not -1 and outside [0, E) */
#define ORC_ERR_BAD_SLOT_EXPERT 2u /* slot_expert outside [0, E) */
#define ORC_ERR_WEIGHT_OVERFLOW 4u /* an expert's plan weights sum to >= 2^32 */

/* ------------------------------------------------------------------ */
/* number formats, from their definitions                              */
/* ------------------------------------------------------------------ */

/* bfloat16: the upper half of an IEEE binary32. */
static double bf16_value(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, 4);
  return (double)f;
}

/* OCP FP8 E4M3 ("E4M3FN"): 1 sign, 4 exponent bits (bias 7), 3 mantissa
 * bits; exponent 0 is subnormal (m/8 * 2^-6); 0x7f / 0xff are NaN; no inf.
 * Largest finite magnitude 1.75 * 2^8 = 448. */
static double e4m3_value(uint8_t c) {
  int s = (c >> 7) & 1, e = (c >> 3) & 15, m = c & 7;
  double v;
  if (e == 15 && m == 7) return NAN;
  if (e == 0) v = ldexp((double)m / 8.0, -6);
  else v = ldexp(1.0 + (double)m / 8.0, e - 7);
  return s ? -v : v;
}

/* Round a double to the nearest bfloat16 value, ties to even (finite
 * inputs).  Done on the double directly, so there is no double rounding. */
static double round_bf16(double x) {
  if (x == 0.0 || !isfinite(x)) return x;
  int e;
  frexp(x, &e); /* |x| in [2^(e-1), 2^e) */
  /* bf16 keeps 8 significant bits: spacing 2^(e-8) (normal range only;
   * the values met here are far from bf16's subnormals). */
  double q = ldexp(1.0, e - 8);
  double r = x / q; /* exact: scaling by a power of two */
  double fl = floor(r);
  double d = r - fl;
  double n;
  if (d > 0.5) n = fl + 1.0;
  else if (d < 0.5) n = fl;
  else n = (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;
  return n * q;
}

/* Nearest E4M3 value to x with ties to even, magnitude saturated at 448. */
static double round_e4m3(double x) {
  double a = fabs(x), best = 0.0;
  int best_code = 0;
  if (a >= 448.0) return x < 0 ? -448.0 : 448.0;
  /* brute force over the 127 non-negative finite codes */
  for (int c = 0; c < 127; c++) {
    double v = e4m3_value((uint8_t)c);
    double d = fabs(v - a), db = fabs(best - a);
    if (c == 0 || d < db || (d == db && (c % 2 == 0))) {
      best = v;
      best_code = c;
    }
  }
  (void)best_code;
  return x < 0 ? -best : best;
}

/* ------------------------------------------------------------------ */
/* counter-based generator: Philox-4x64 with 10 rounds (Salmon, Moraes,  */
/* Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3", SC 2011).  */
/* Each round multiplies counter words 0 and 2 by the round constants    */
/* into 128-bit products, permutes and XORs in the key; the key is       */
/* bumped by the Weyl constants between rounds.                          */
/* ------------------------------------------------------------------ */

void oracle_philox4x64_10(const uint64_t ctr[4], const uint64_t key[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3], k0 = key[0], k1 = key[1];
  for (int r = 0; r < 10; r++) {
    unsigned __int128 p0 = (unsigned __int128)c0 * M0, p1 = (unsigned __int128)c2 * M1;
    uint64_t hi0 = (uint64_t)(p0 >> 64), lo0 = (uint64_t)p0, hi1 = (uint64_t)(p1 >> 64), lo1 = (uint64_t)p1;
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += W0;
    k1 += W1;
  }
  out[0] = c0;
  out[1] = c1;
  out[2] = c2;
  out[3] = c3;
}

/* ------------------------------------------------------------------ */
/* stage 1: dispatch                                                   */
/* ------------------------------------------------------------------ */

/*
 * Inputs
 *   T, T_valid, K, E, S, M     batch rows, real rows, top-k, logical experts,
 *                              local slots, M-tile.
 *   topk_ids   [T*K]           expert id of pair p = t*K + k; -1 = no expert.
 *   slot_expert [S]            logical expert held by local slot s.
 *   slot_weight [S]            integer share weight of slot s.
 *   remote_weight [E]          share weight kept by replicas on other GPUs.
 *   remote_replicas [E]        number of replicas on other GPUs.
 * Outputs
 *   expert_counts [E]          n_e over valid pairs (all experts).
 *   slot_counts [S]            c_s.
 *   slot_offsets [S+1]         exclusive prefix sum of P_s = M*ceil(c_s/M).
 *   row_token [slot_offsets[S]]  token of each row, -1 on padding rows.
 *   pair_row [T*K]             row of each pair, -1 if not placed locally.
 *   cum_counts [E] (nullable)  (cum + n_e) mod 2^32.
 *   flags                      bit 0: tile-aware split (below); bit 1: sampled
 *                              replicas (below; bit 0 is then ignored).
 *   seed                       key of the generator (sampled replicas).
 * Returns the error bits.
 *
 * Sampled replicas (Sec. 4.4: the deployed kernel samples one replica per
 * pair from the renormalised table row).  Pair p = t*K + k of expert e draws
 * r = word 0 of Philox-4x64-10 at counter (p, 0, 0, 0) with key (seed, 0),
 * u = floor(hi32(r) * W / 2^32) in [0, W), and goes to the first entry j
 * with u < C_j (entries and weights as in the split, the zero-sum fallback
 * included).  The rows of a slot hold its pairs in ascending p.
 *
 * Tile-aware split (Sec. 2.2 after Eq. 2: the solver snaps partial splits
 * to tile boundaries so that an expert's rows fill whole M-tiles).  Reading:
 * every boundary floor(n_e C_j / W) other than n_e itself moves to the
 * nearest multiple of M (halves round up), capped at n_e; the expert's last
 * entry takes the remainder.  With M = 1 this is the plain split.
 */
uint32_t oracle_dispatch(int T, int T_valid, int K, int E, int S, int M, const int32_t* topk_ids,
                         const int32_t* slot_expert, const uint32_t* slot_weight,
                         const uint32_t* remote_weight, const int32_t* remote_replicas,
                         int32_t* expert_counts, int32_t* slot_counts, int32_t* slot_offsets,
                         int32_t* row_token, int32_t* pair_row, uint32_t* cum_counts, int flags, uint64_t seed) {
  const int snap_tiles = (flags & 1) && !(flags & 2), sample = (flags & 2) != 0;
  uint32_t err = 0;
  int P = T * K;

  /* 1-2. valid pairs and their per-expert counts; graph-padding rows
   * (t >= T_valid) are masked out. */
  for (int e = 0; e < E; e++) expert_counts[e] = 0;
  for (int p = 0; p < P; p++) pair_row[p] = -1;
  for (int t = 0; t < T_valid; t++)
    for (int k = 0; k < K; k++) {
      int id = topk_ids[t * K + k];
      if (id == -1) continue;
      if (id < 0 || id >= E) {
        err |= ORC_ERR_BAD_ID;
        continue;
      }
      expert_counts[id]++;
    }
  for (int s = 0; s < S; s++)
    if (slot_expert[s] < 0 || slot_expert[s] >= E) err |= ORC_ERR_BAD_SLOT_EXPERT;

  /* 3. per expert: split n_e over its entries (local slots in ascending
   * slot order, then one REMOTE entry), cumulative-floor boundaries. */
  int32_t* slot_lo = (int32_t*)calloc((size_t)S + 1, sizeof(int32_t));
  for (int s = 0; s < S; s++) slot_counts[s] = 0;
  int32_t* ent_slot = (int32_t*)malloc(((size_t)S + 1) * sizeof(int32_t));
  uint64_t* ent_w = (uint64_t*)malloc(((size_t)S + 1) * sizeof(uint64_t));
  int64_t* ent_b = (int64_t*)malloc(((size_t)S + 2) * sizeof(int64_t));
  int32_t* pair_slot = (int32_t*)malloc(((size_t)P + 1) * sizeof(int32_t)); /* sampled: slot of each pair */
  for (int p = 0; p < P; p++) pair_slot[p] = -1;
  for (int e = 0; e < E; e++) {
    int nent = 0;
    for (int s = 0; s < S; s++)
      if (slot_expert[s] == e) {
        ent_slot[nent] = s;
        ent_w[nent] = slot_weight[s];
        nent++;
      }
    int has_remote = remote_weight[e] > 0 || remote_replicas[e] > 0;
    if (has_remote) {
      ent_slot[nent] = -1;
      ent_w[nent] = remote_weight[e];
      nent++;
    }
    if (nent == 0) continue;
    uint64_t W = 0;
    for (int j = 0; j < nent; j++) W += ent_w[j];
    int uniform = (W == 0);
    if (W >= ((uint64_t)1 << 32)) {
      err |= ORC_ERR_WEIGHT_OVERFLOW;
      uniform = 1;
    }
    if (uniform) {
      /* renormalising a zero (or unusable) row: uniform over the replicas
       * that hold the expert -- one per local slot, remote_replicas[e]
       * for the others. */
      W = 0;
      for (int j = 0; j < nent; j++) {
        ent_w[j] = (ent_slot[j] >= 0) ? 1u : (uint64_t)(remote_replicas[e] > 0 ? remote_replicas[e] : 0);
        W += ent_w[j];
      }
    }
    if (sample) {
      /* one draw per valid pair of the expert, entry by cumulative weight */
      for (int p = 0; p < T_valid * K; p++) {
        if (topk_ids[p] != e) continue;
        const uint64_t ctr[4] = {(uint64_t)p, 0, 0, 0}, key[2] = {seed, 0};
        uint64_t rnd[4];
        oracle_philox4x64_10(ctr, key, rnd);
        const uint64_t u = ((rnd[0] >> 32) * W) >> 32;
        uint64_t Cj = 0;
        for (int j = 0; j < nent; j++) {
          Cj += ent_w[j];
          if (u < Cj) {
            if (ent_slot[j] >= 0) {
              pair_slot[p] = ent_slot[j];
              slot_counts[ent_slot[j]]++;
            }
            break;
          }
        }
      }
      continue;
    }
    uint64_t n = (uint64_t)expert_counts[e];
    uint64_t C = 0;
    ent_b[0] = 0;
    for (int j = 0; j < nent; j++) {
      C += ent_w[j];
      int64_t b = (int64_t)((n * C) / W);
      if (snap_tiles && b != (int64_t)n) {
        int64_t q = (b + M / 2) / M * M;
        b = q < (int64_t)n ? q : (int64_t)n;
      }
      ent_b[j + 1] = b;
    }
    for (int j = 0; j < nent; j++)
      if (ent_slot[j] >= 0) {
        slot_counts[ent_slot[j]] = (int32_t)(ent_b[j + 1] - ent_b[j]);
        slot_lo[ent_slot[j]] = (int32_t)ent_b[j];
      }
  }

  /* 5. padded group sizes and their exclusive prefix sum. */
  slot_offsets[0] = 0;
  for (int s = 0; s < S; s++) {
    int c = slot_counts[s];
    int Ps = ((c + M - 1) / M) * M;
    slot_offsets[s + 1] = slot_offsets[s] + Ps;
  }
  for (int r = 0; r < slot_offsets[S]; r++) row_token[r] = -1;

  /* 4+6. stable rank of each pair within its expert (ascending p), rank ->
   * entry, entry -> row.  Sampled: the rows of a slot in ascending p. */
  if (sample) {
    for (int s = 0; s < S; s++) {
      int r = 0;
      for (int p = 0; p < T_valid * K; p++)
        if (pair_slot[p] == s) {
          const int row = slot_offsets[s] + r++;
          pair_row[p] = row;
          row_token[row] = p / K;
        }
    }
  }
  for (int e = 0; e < E && !sample; e++) {
    int r = 0;
    for (int p = 0; p < T_valid * K; p++) {
      if (topk_ids[p] != e) continue;
      for (int s = 0; s < S; s++)
        if (slot_expert[s] == e && r >= slot_lo[s] && r < slot_lo[s] + slot_counts[s]) {
          int row = slot_offsets[s] + (r - slot_lo[s]);
          pair_row[p] = row;
          row_token[row] = p / K;
        }
      r++;
    }
  }

  /* 8. cumulative counter, modulo 2^32. */
  if (cum_counts)
    for (int e = 0; e < E; e++) cum_counts[e] = cum_counts[e] + (uint32_t)expert_counts[e];

  free(slot_lo);
  free(ent_slot);
  free(ent_w);
  free(ent_b);
  free(pair_slot);
  return err;
}

/* ------------------------------------------------------------------ */
/* stages 2 + 3: expert FFN and routing-weighted combine               */
/* ------------------------------------------------------------------ */

/* dtype: 0 = bf16 (uint16 storage), 1 = fp8 e4m3 (uint8 storage) with
 * scales, 2 = fp8 e4m3 whose scales are powers of two (UE8M0; the paper's
 * note that newer hardware requires them, App. "Multi-node bring-up
 * notes"): the same values, only the re-quantisation of h picks its scale
 * differently (below); 1 or 2
 * fp32 scales: activations 1 x 128 along the contraction, weights 128 x 128
 * blocks (the gate/up matrix [2I, H] is blocked as one matrix). */
static double x_at(int dtype, const void* x, const float* xs, int H, int t, int h) {
  if (dtype == 0) return bf16_value(((const uint16_t*)x)[(size_t)t * H + h]);
  return e4m3_value(((const uint8_t*)x)[(size_t)t * H + h]) * (double)xs[(size_t)t * (H / 128) + h / 128];
}

static double w_at(int dtype, const void* w, const float* ws, size_t slot_elems, int rows, int cols, int s,
                   int r, int c) {
  size_t idx = (size_t)s * slot_elems + (size_t)r * cols + c;
  if (dtype == 0) return bf16_value(((const uint16_t*)w)[idx]);
  size_t sidx = (size_t)s * (size_t)(rows / 128) * (cols / 128) + (size_t)(r / 128) * (cols / 128) + c / 128;
  return e4m3_value(((const uint8_t*)w)[idx]) * (double)ws[sidx];
}

/* One pair's expert FFN: o = W2_s (silu(W_gate,s x) * (W_up,s x)), x given in
 * fp64 (already dequantised).  hv [I] is scratch; o [H] receives the result.
 * mode 1 rounds h (bf16, or e4m3 with 1 x 128 scales amax/448) and o (bf16). */
static void ffn_one(int H, int I, int dtype, int mode, const double* xv, int s, const void* w13,
                    const float* w13_scale, const void* w2, const float* w2_scale, double* hv, double* o) {
  size_t w13_elems = (size_t)2 * I * H, w2_elems = (size_t)H * I;
  /* gate/up projections and SwiGLU: h = silu(g) * u, silu(g) = g/(1+e^-g) */
  for (int i = 0; i < I; i++) {
    double g = 0.0, u = 0.0;
    for (int h = 0; h < H; h++) {
      g += w_at(dtype, w13, w13_scale, w13_elems, 2 * I, H, s, i, h) * xv[h];
      u += w_at(dtype, w13, w13_scale, w13_elems, 2 * I, H, s, I + i, h) * xv[h];
    }
    hv[i] = g / (1.0 + exp(-g)) * u;
  }
  if (mode == 1) {
    if (dtype == 0) {
      for (int i = 0; i < I; i++) hv[i] = round_bf16(hv[i]);
    } else {
      /* 1 x 128 block quantisation: scale = amax / 448 (dtype 2: the
       * smallest power of two at least amax / 448), q = e4m3(h / scale) */
      for (int b = 0; b < I / 128; b++) {
        double amax = 0.0;
        for (int i = b * 128; i < b * 128 + 128; i++) amax = fmax(amax, fabs(hv[i]));
        double sc = amax > 0.0 ? amax / 448.0 : 1.0;
        if (dtype == 2 && amax > 0.0) {
          int ex;
          const double f = frexp(sc, &ex); /* sc = f 2^ex, f in [0.5, 1) */
          sc = ldexp(1.0, f == 0.5 ? ex - 1 : ex);
        }
        for (int i = b * 128; i < b * 128 + 128; i++) hv[i] = round_e4m3(hv[i] / sc) * sc;
      }
    }
  }
  /* down projection */
  for (int j = 0; j < H; j++) {
    double acc = 0.0;
    for (int i = 0; i < I; i++) acc += w_at(dtype, w2, w2_scale, w2_elems, H, I, s, j, i) * hv[i];
    o[j] = (mode == 1) ? round_bf16(acc) : acc;
  }
}

/*
 *   x [T, H], x_scale [T, H/128] (fp8 only)
 *   w13 [S, 2I, H] rows 0..I-1 = gate, I..2I-1 = up; w13_scale [S, 2I/128, H/128]
 *   w2  [S, H, I];                                   w2_scale  [S, H/128, I/128]
 *   topk_w [T*K] fp32 routing weights
 *   pair_slot [T*K]  local slot of each pair, -1 = not local
 *   token_sel [T]    nonzero = compute this token's row of y (others untouched)
 *   y [T, H] double  output: y[t] = sum over k ascending of w[t,k] * o_{t,k}
 *                    over the token's local pairs (mode 1: rounded to bf16)
 */
void oracle_moe(int T, int K, int H, int I, int S, int dtype, int mode, const void* x, const float* x_scale,
                const void* w13, const float* w13_scale, const void* w2, const float* w2_scale,
                const float* topk_w, const int32_t* pair_slot, const uint8_t* token_sel, double* y) {
  (void)S;
#pragma omp parallel for schedule(dynamic, 1)
  for (int t = 0; t < T; t++) {
    if (!token_sel[t]) continue;
    double* xv = (double*)malloc(sizeof(double) * (size_t)H);
    double* hv = (double*)malloc(sizeof(double) * (size_t)I);
    double* o = (double*)malloc(sizeof(double) * (size_t)H);
    double* yt = y + (size_t)t * H;
    for (int j = 0; j < H; j++) yt[j] = 0.0;
    for (int h = 0; h < H; h++) xv[h] = x_at(dtype, x, x_scale, H, t, h);
    for (int k = 0; k < K; k++) {
      int s = pair_slot[t * K + k];
      if (s < 0) continue;
      ffn_one(H, I, dtype, mode, xv, s, w13, w13_scale, w2, w2_scale, hv, o);
      double wk = (double)topk_w[t * K + k];
      for (int j = 0; j < H; j++) yt[j] += wk * o[j];
    }
    if (mode == 1)
      for (int j = 0; j < H; j++) yt[j] = round_bf16(yt[j]);
    free(xv);
    free(hv);
    free(o);
  }
}

/* Stage 2 alone: o for each selected (token, slot) row.  tok [R], slot [R];
 * out [R, H] double.  Rows with slot < 0 are left untouched. */
void oracle_ffn_rows(int R, int H, int I, int dtype, int mode, const void* x, const float* x_scale,
                     const int32_t* tok, const int32_t* slot, const void* w13, const float* w13_scale,
                     const void* w2, const float* w2_scale, double* out) {
#pragma omp parallel for schedule(dynamic, 1)
  for (int r = 0; r < R; r++) {
    if (slot[r] < 0) continue;
    double* xv = (double*)malloc(sizeof(double) * (size_t)H);
    double* hv = (double*)malloc(sizeof(double) * (size_t)I);
    for (int h = 0; h < H; h++) xv[h] = x_at(dtype, x, x_scale, H, tok[r], h);
    ffn_one(H, I, dtype, mode, xv, slot[r], w13, w13_scale, w2, w2_scale, hv, out + (size_t)r * H);
    free(xv);
    free(hv);
  }
}

/* Stage 3 alone: y[t] = sum over k ascending with pair_row >= 0 of
 * w[t,k] * y_perm[pair_row[t,k]] (y_perm given as bf16 bits), for t < T_valid;
 * zero elsewhere.  y [T, H] double. */
void oracle_combine(int T, int T_valid, int K, int H, const int32_t* pair_row, const float* topk_w,
                    const uint16_t* y_perm, double* y) {
  for (int t = 0; t < T; t++)
    for (int j = 0; j < H; j++) {
      double acc = 0.0;
      if (t < T_valid)
        for (int k = 0; k < K; k++) {
          int r = pair_row[t * K + k];
          if (r < 0) continue;
          acc += (double)topk_w[t * K + k] * bf16_value(y_perm[(size_t)r * H + j]);
        }
      y[(size_t)t * H + j] = acc;
    }
}

/* exported helpers so the tests can pin the number formats themselves */
double oracle_bf16_value(uint16_t b) { return bf16_value(b); }
double oracle_e4m3_value(uint8_t c) { return e4m3_value(c); }
double oracle_round_bf16(double x) { return round_bf16(x); }
double oracle_round_e4m3(double x) { return round_e4m3(x); }
