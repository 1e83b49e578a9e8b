/* Randomised check of the oracle's C coder (oracle/coder.c), built with
 * AddressSanitizer and UndefinedBehaviorSanitizer by tests/test_host_fuzz.py:
 * tables quantised from random log-softmax rows keep their invariants
 * (cumulative, each alphabet bin at least 1, total T), random symbol strings
 * encode and decode back, and random byte vectors serialise and deserialise
 * back for every grouping.  Returns 0 when every check holds. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int64_t orc_num_tokens(int64_t, int32_t, int32_t, int32_t);
int64_t orc_serialize(const uint8_t*, int64_t, int32_t, int32_t, int32_t, const int32_t*, int32_t,
                      int32_t, int32_t*, uint8_t*);
int orc_deserialize(const uint8_t*, int64_t, int64_t, int32_t, int32_t, int32_t, int32_t, uint8_t*);
void orc_quantize(const float*, int32_t, int32_t, uint32_t, uint32_t*);
int64_t orc_ac_encode(const uint32_t*, int32_t, const uint8_t*, int64_t, uint8_t*, uint64_t);
void orc_ac_decode(const uint32_t*, int32_t, int64_t, const uint8_t*, uint64_t, uint8_t*);

static uint64_t st;
static uint64_t rnd(void) {  /* splitmix64 */
  uint64_t z = (st += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}
static double unif(void) { return (rnd() >> 11) * (1.0 / 9007199254740992.0); }

#define FAIL(...) do { printf(__VA_ARGS__); printf("\n"); return 1; } while (0)

int main(int argc, char** argv) {
  st = argc > 1 ? strtoull(argv[1], 0, 10) : 1;
  for (int it = 0; it < 400; it++) {
    const int na = 17 + (int)(rnd() % 2), nsym = na + 1, renorm = (int)(rnd() % 2);
    const uint32_t T = (rnd() % 2) ? (1u << 16) : (1u << 24);
    const int n = 1 + (int)(rnd() % 600);
    uint32_t* cdf = malloc(sizeof(uint32_t) * n * (nsym + 1));
    uint8_t* sym = malloc(n);
    const double scale = 0.1 + 30.0 * unif();
    for (int r = 0; r < n; r++) {
      /* log-softmax over the alphabet (renorm) or over a larger vocabulary */
      float lp[18];
      double z[18], m = -1e300, se = 0.0;
      for (int a = 0; a < na; a++) { z[a] = scale * (unif() - 0.5); if (z[a] > m) m = z[a]; }
      const double rest = renorm ? 0.0 : exp(scale * (unif() - 0.5) - m) * (1 + rnd() % 32000);
      for (int a = 0; a < na; a++) se += exp(z[a] - m);
      se += rest;
      for (int a = 0; a < na; a++) lp[a] = (float)(z[a] - m - log(se));
      uint32_t* c = cdf + (size_t)r * (nsym + 1);
      orc_quantize(lp, na, renorm, T, c);
      if (c[0] != 0 || c[nsym] != T) FAIL("table ends %u %u", c[0], c[nsym]);
      for (int k = 0; k < na; k++)
        if (c[k + 1] < c[k] + 1) FAIL("alphabet bin %d empty", k);
      if (c[nsym] < c[na]) FAIL("escape bin negative");
      if (!renorm && c[nsym] == c[na]) FAIL("escape bin empty without renorm");
      sym[r] = (uint8_t)(rnd() % na);
    }
    const uint64_t cap = 64 + (uint64_t)n * 8;
    uint8_t* out = calloc(cap, 1);
    const int64_t bits = orc_ac_encode(cdf, nsym, sym, n, out, cap);
    if (bits < 0) FAIL("encode failed");
    uint8_t* back = malloc(n);
    orc_ac_decode(cdf, nsym, n, out, (uint64_t)bits, back);
    if (memcmp(back, sym, n)) FAIL("decode mismatch");
    free(cdf); free(sym); free(out); free(back);
  }
  int32_t hex[16];
  for (int i = 0; i < 16; i++) hex[i] = i < 10 ? 48 + i : 87 + i;
  for (int it = 0; it < 2000; it++) {
    const int32_t bpv = (int32_t[]){1, 2, 4}[rnd() % 3], bpg = (int32_t)(rnd() % 9);
    const int32_t msb = (int32_t)(rnd() % 2), two = (int32_t)(rnd() % 2);
    const int64_t nv = (int64_t)(rnd() % 40);
    const int64_t nt = orc_num_tokens(nv, bpv, bpg, two ? 2 : 1);
    uint8_t* v = malloc(nv * bpv + 1);
    for (int64_t i = 0; i < nv * bpv; i++) v[i] = (uint8_t)rnd();
    int32_t* tok = malloc(sizeof(int32_t) * (nt + 1));
    uint8_t* s = malloc(nt + 1);
    if (orc_serialize(v, nv, bpv, bpg, msb, hex, 32, two ? 44 : -1, tok, s) != nt) FAIL("token count");
    uint8_t* w = malloc(nv * bpv + 1);
    if (orc_deserialize(s, nt, nv, bpv, bpg, msb, two ? 2 : 1, w)) FAIL("deserialize rejected");
    if (memcmp(v, w, nv * bpv)) FAIL("serialise round trip");
    free(v); free(tok); free(s); free(w);
  }
  printf("oracle fuzz ok\n");
  return 0;
}
