/*
 * tracegen.c -- seeded synthetic event traces for the batched claim-arbitration replay.
 *
 * Input generation only: this file draws events and lays out pool descriptors; it holds none of
 * the replay's arithmetic and never simulates a pool.  Both the HIP library's tests and the
 * oracle's tests consume the bytes it writes.
 *
 * Random numbers: xoshiro256** (Blackman and Vigna, "Scrambled linear pseudorandom number
 * generators", 2018), one stream per (config, pool), seeded through SplitMix64 (Steele, Lea and
 * Flood, 2014) from seed0 ^ (config << 32) ^ pool.  A uniform double takes the top 53 bits.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct { uint64_t s[4]; } rng_t;

static uint64_t splitmix64(uint64_t* x) {
  uint64_t z = (*x += 0x9e3779b97f4a7c15ULL);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ULL;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebULL;
  return z ^ (z >> 31);
}

static uint64_t rotl(uint64_t x, int k) { return (x << k) | (x >> (64 - k)); }

static uint64_t next_u64(rng_t* r) {
  uint64_t* s = r->s;
  uint64_t out = rotl(s[1] * 5, 7) * 9;
  uint64_t t = s[1] << 17;
  s[2] ^= s[0];
  s[3] ^= s[1];
  s[1] ^= s[2];
  s[0] ^= s[3];
  s[2] ^= t;
  s[3] = rotl(s[3], 45);
  return out;
}

static void seed_rng(rng_t* r, uint64_t seed) {
  uint64_t x = seed;
  for (int i = 0; i < 4; i++) r->s[i] = splitmix64(&x);
}

static double unit(rng_t* r) { return (double)(next_u64(r) >> 11) * (1.0 / 9007199254740992.0); }

static int32_t uniform_int(rng_t* r, int32_t a, int32_t b) {
  int64_t v = a + (int64_t)floor(unit(r) * (double)((int64_t)b - a + 1));
  if (v > b) v = b;
  return (int32_t)v;
}

static int32_t loguniform_int(rng_t* r, int32_t a, int32_t b) {
  double la = log((double)a), lb = log((double)b + 1.0);
  int64_t v = (int64_t)floor(exp(la + unit(r) * (lb - la)));
  if (v < a) v = a;
  if (v > b) v = b;
  return (int32_t)v;
}

/* Parameters of one synthetic configuration (all block counts in blocks). */
typedef struct {
  int32_t cfg_id;
  int32_t usable_blocks, n_events;
  int32_t mix[6];          /* per-mille of PREFILL, EXTEND, CLAIM, FINISH, RELEASE, DEMOTE      */
  int32_t prefill_dist;    /* 0 uniform, 1 log-uniform                                          */
  int32_t prefill_min, prefill_max;
  int32_t chain_pick;      /* 0: prefills private, claims on a fresh chain each;
                              1: Zipf over n_chains; 2: uniform over n_chains                    */
  int32_t n_chains;
  int32_t chain_len_min, chain_len_max; /* per pool, per chain                                   */
  int32_t claim_len;       /* 0: L = chain length; 1: uniform [lmin,lmax]; 2: log-uniform        */
  int32_t claim_len_min, claim_len_max;
  int32_t claim_thresh;    /* 0: T = L; 1: T uniform in [ceil(L/2), L]                           */
  int32_t hard_permille;
  int32_t prio_max;
  int32_t dur_min, dur_max; /* 0,0 = no expiry                                                    */
  int32_t extend_k;
  int32_t claim_cap;       /* >0: at most this many outstanding claims (a CLAIM drawn at the cap
                              becomes a RELEASE)                                                 */
  int32_t max_live_claims, max_live_requests; /* <= 0: the pool's own CLAIM / PREFILL count      */
  int32_t retry_permille;  /* > 0: share of RETRY events, drawn before the mix                   */
  int32_t defer_limit;     /* the pools' defer limit (0 = no deferral)                           */
  int32_t mode;            /* < 0: policy = pool index mod 4; else this mode for every pool       */
  int32_t demotable_permille; /* > 0: share of CLAIM events marked demotable (extra draw only then) */
  int32_t offloadable_permille; /* > 0: share of CLAIM events marked offloadable (extra draw only
                                   then)                                                         */
  int32_t offload_blocks;  /* the pools' second-tier capacity in blocks (0 = none)              */
  double zipf_s;
  uint64_t seed0;
} gen_params;

enum { EV_PREFILL = 0, EV_EXTEND = 1, EV_CLAIM = 2, EV_FINISH = 3, EV_RELEASE = 4, EV_DEMOTE = 5,
       EV_RETRY = 7 };

/* Draw the events of pools [first_pool, first_pool + n_pools).
 * desc: 16 int32 per pool; events: n_pools * n_events * 4 int32.
 * Returns the total number of claim slots (CLAIM events), or -1 on bad parameters. */
int64_t rkc_tracegen(const gen_params* g, int64_t first_pool, int32_t n_pools, int32_t* desc,
                     int32_t* events) {
  if (!g || g->n_events < 0 || g->usable_blocks < 1 || n_pools < 0) return -1;
  int32_t nch = g->n_chains > 0 ? g->n_chains : 0;
  double* zcdf = NULL;
  int32_t* clen = (int32_t*)malloc((size_t)(nch > 0 ? nch : 1) * sizeof(int32_t));
  if (g->chain_pick == 1 && nch > 0) {
    zcdf = (double*)malloc((size_t)nch * sizeof(double));
    double acc = 0;
    for (int32_t k = 0; k < nch; k++) { acc += pow((double)(k + 1), -g->zipf_s); zcdf[k] = acc; }
    for (int32_t k = 0; k < nch; k++) zcdf[k] /= acc;
  }
  int32_t cum[6];
  for (int i = 0, a = 0; i < 6; i++) { a += g->mix[i]; cum[i] = a; }
  int64_t slots = 0;
  for (int32_t i = 0; i < n_pools; i++) {
    int64_t pool = first_pool + i;
    rng_t r;
    seed_rng(&r, g->seed0 ^ ((uint64_t)(uint32_t)g->cfg_id << 32) ^ (uint64_t)pool);
    for (int32_t c = 0; c < nch; c++) clen[c] = uniform_int(&r, g->chain_len_min, g->chain_len_max);
    int32_t* ev = events + (size_t)4 * (size_t)g->n_events * (size_t)i;
    int32_t n_claims = 0, n_prefill = 0, outstanding = 0;
    for (int32_t t = 0; t < g->n_events; t++) {
      int32_t* e = ev + 4 * (size_t)t;
      if (g->retry_permille > 0 && uniform_int(&r, 0, 999) < g->retry_permille) {
        e[0] = EV_RETRY; e[1] = e[2] = e[3] = 0;
        continue;
      }
      int32_t u = uniform_int(&r, 0, cum[5] - 1), type = 0;
      while (type < 5 && u >= cum[type]) type++;
      if (type == EV_CLAIM && g->claim_cap > 0 && outstanding >= g->claim_cap) type = EV_RELEASE;
      e[0] = e[1] = e[2] = e[3] = 0;
      if (type == EV_PREFILL) {
        int32_t S = g->prefill_dist ? loguniform_int(&r, g->prefill_min, g->prefill_max)
                                    : uniform_int(&r, g->prefill_min, g->prefill_max);
        int32_t c = -1, P = 0;
        if (g->chain_pick == 1 || g->chain_pick == 2) {
          if (g->chain_pick == 1) {
            double x = unit(&r);
            int32_t lo = 0, hi = nch - 1;
            while (lo < hi) { int32_t m = (lo + hi) / 2; if (zcdf[m] > x) hi = m; else lo = m + 1; }
            c = lo;
          } else {
            c = uniform_int(&r, 0, nch - 1);
          }
          P = S < clen[c] ? S : clen[c];
        }
        e[0] = EV_PREFILL; e[1] = S; e[2] = c; e[3] = P;
        n_prefill++;
      } else if (type == EV_EXTEND) {
        e[0] = EV_EXTEND; e[1] = g->extend_k; e[2] = (int32_t)(uint32_t)next_u64(&r);
      } else if (type == EV_CLAIM) {
        int32_t c;
        if (g->chain_pick == 1) {
          double x = unit(&r);
          int32_t lo = 0, hi = nch - 1;
          while (lo < hi) { int32_t m = (lo + hi) / 2; if (zcdf[m] > x) hi = m; else lo = m + 1; }
          c = lo;
        } else if (g->chain_pick == 2) {
          c = uniform_int(&r, 0, nch - 1);
        } else {
          c = n_claims; /* a fresh chain per claim */
        }
        int32_t L;
        if (g->claim_len == 0) L = clen[c];
        else if (g->claim_len == 1) L = uniform_int(&r, g->claim_len_min, g->claim_len_max);
        else L = loguniform_int(&r, g->claim_len_min, g->claim_len_max);
        int32_t T = g->claim_thresh ? uniform_int(&r, (L + 1) / 2, L) : L;
        int32_t hard = (int32_t)(uniform_int(&r, 0, 999) < g->hard_permille);
        int32_t prio = uniform_int(&r, 0, g->prio_max);
        int32_t dur = g->dur_max > 0 ? uniform_int(&r, g->dur_min, g->dur_max) : 0;
        int32_t dem = g->demotable_permille > 0 && uniform_int(&r, 0, 999) < g->demotable_permille;
        int32_t off = g->offloadable_permille > 0 && uniform_int(&r, 0, 999) < g->offloadable_permille;
        e[0] = (int32_t)((uint32_t)EV_CLAIM | ((uint32_t)hard << 4) | ((uint32_t)prio << 5) |
                         ((uint32_t)dem << 7) | ((uint32_t)off << 9) | ((uint32_t)dur << 16));
        e[1] = L; e[2] = c; e[3] = T;
        n_claims++;
        outstanding++;
      } else {
        e[0] = type;
        e[1] = (int32_t)(uint32_t)next_u64(&r);
        if (type == EV_RELEASE && outstanding > 0) outstanding--;
      }
    }
    int32_t* d = desc + 16 * (size_t)i;
    int64_t ev_off = (int64_t)g->n_events * (first_pool + i) - (int64_t)g->n_events * first_pool;
    d[0] = g->usable_blocks;
    d[1] = g->mode >= 0 ? g->mode : (int32_t)(pool % 4);
    d[2] = g->n_events;
    d[3] = g->chain_pick == 0 ? n_claims : nch;
    d[4] = g->max_live_claims > 0 ? g->max_live_claims : n_claims;
    d[5] = g->max_live_requests > 0 ? g->max_live_requests : n_prefill;
    d[6] = n_claims;
    d[7] = g->defer_limit;
    d[8] = g->offload_blocks;
    d[9] = d[10] = d[11] = 0;
    d[12] = (int32_t)(uint32_t)(uint64_t)ev_off;
    d[13] = (int32_t)((uint64_t)ev_off >> 32);
    d[14] = (int32_t)(uint32_t)(uint64_t)slots;
    d[15] = (int32_t)((uint64_t)slots >> 32);
    slots += n_claims;
  }
  free(zcdf);
  free(clen);
  return slots;
}
