/*
 * LM-GC reference coder -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, obviously-correct C for the integer parts of LM-GC:
 *   - hex serialisation of values and its inverse      (Sec. 4, "Serialization")
 *   - quantisation of per-position log-probabilities
 *     into an integer frequency table / CDF             (Sec. 4, "Compression":
 *                                                        the LM's distribution is
 *                                                        the coder's model)
 *   - a Witten-Neal-Cleary binary arithmetic coder      (Sec. 3, "Arithmetic coding")
 *
 * Only the tests, the smoke check and the benchmark's CPU-baseline leg may load
 * this file's library.  It shares no code with the GPU library.
 *
 * Readings of the paper used here (it is silent on them):
 *   - nibble order: most significant nibble first (msb_first=1), or the bytes
 *     in memory (little-endian) order with the high nibble of each byte first;
 *   - a separator follows every group of bytes_per_group bytes, including the
 *     last (possibly partial) group; bytes_per_group=0 means no separator;
 *   - bins 0..15 are the hex digits, bin 16 the separator (bin 17 a second
 *     separator token when the separator is two characters), then an escape
 *     bin that holds the probability of every other vocabulary entry and is
 *     never coded; A = 17 or 18 alphabet symbols;
 *   - frequencies: f_a = 1 + floor(exp(lp_a) * (T - (A + 1))), computed in
 *     double from the float32 log-probability; if the A frequencies sum past
 *     T-1 the largest (lowest index on ties) gives up the excess; the escape
 *     bin takes T - sum;
 *   - renormalised tables (the LM's distribution restricted to the alphabet
 *     and renormalised over it, so the escape bin is empty): lp_a is the
 *     log-probability within the alphabet, f_a = 1 + floor(exp(lp_a) * (T - A)),
 *     the largest f_a (lowest index on ties) takes T - sum, whatever its
 *     sign, and the escape bin has width 0 (cdf[A] = cdf[A+1] = T), which
 *     codes exactly as an A-bin table;
 *   - coder: 62-bit code values, E1/E2/E3 renormalisation with pending bits,
 *     flush = pending+1 then one bit chosen by low < quarter; bits are packed
 *     most significant first, the last byte padded with zero bits; the
 *     decoder reads zero bits past the end of the stream.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORC_NSYM_MAX 19 /* 16 hex digits + up to two separator tokens + escape */

/* ------------------------------------------------------------------------ */
/* Serialisation                                                             */
/* ------------------------------------------------------------------------ */

/* Number of tokens a vector of n values serialises to (nsep separator
 * tokens after each group). */
int64_t orc_num_tokens(int64_t n_values, int32_t bytes_per_value,
                       int32_t bytes_per_group, int32_t nsep) {
  int64_t nbytes = n_values * (int64_t)bytes_per_value;
  int64_t ngroups = 0;
  if (bytes_per_group > 0) ngroups = (nbytes + bytes_per_group - 1) / bytes_per_group;
  return 2 * nbytes + ngroups * nsep;
}

/* Byte k (0-based, in emission order) of value i. */
static uint8_t value_byte(const uint8_t* values, int64_t i, int32_t k,
                          int32_t bpv, int32_t msb_first) {
  int32_t mem = msb_first ? (bpv - 1 - k) : k; /* little-endian storage */
  return values[i * bpv + mem];
}

/*
 * Serialise n values (raw little-endian bytes, bpv bytes each) into a token
 * stream.  tokens[t] gets the token id, sym[t] the coder bin: 0..15 digits,
 * 16 the separator sep_id, 17 the second separator sep2_id (only when
 * sep2_id >= 0; the comma-and-space separator of the paper's H_c+s).
 * Returns the number of tokens written.
 */
int64_t orc_serialize(const uint8_t* values, int64_t n_values, int32_t bpv,
                      int32_t bpg, int32_t msb_first, const int32_t* hex_ids,
                      int32_t sep_id, int32_t sep2_id, int32_t* tokens, uint8_t* sym) {
  int64_t t = 0;
  int64_t byte_no = 0; /* bytes emitted since the stream start */
  int64_t nbytes = n_values * (int64_t)bpv;
  for (int64_t i = 0; i < n_values; i++) {
    for (int32_t k = 0; k < bpv; k++) {
      uint8_t b = value_byte(values, i, k, bpv, msb_first);
      uint8_t hi = (uint8_t)(b >> 4), lo = (uint8_t)(b & 15);
      tokens[t] = hex_ids[hi]; sym[t] = hi; t++;
      tokens[t] = hex_ids[lo]; sym[t] = lo; t++;
      byte_no++;
      if (bpg > 0 && (byte_no % bpg == 0 || byte_no == nbytes)) {
        tokens[t] = sep_id; sym[t] = 16; t++;
        if (sep2_id >= 0) { tokens[t] = sep2_id; sym[t] = 17; t++; }
      }
    }
  }
  return t;
}

/*
 * Inverse of orc_serialize on coder bins.  Checks the structure (digits where
 * digits belong, separators where separators belong, exact length).
 * Returns 0 on success, -1 if the stream is malformed.
 */
int orc_deserialize(const uint8_t* sym, int64_t n_tokens, int64_t n_values,
                    int32_t bpv, int32_t bpg, int32_t msb_first, int32_t nsep,
                    uint8_t* values) {
  if (orc_num_tokens(n_values, bpv, bpg, nsep) != n_tokens) return -1;
  int64_t t = 0, byte_no = 0, nbytes = n_values * (int64_t)bpv;
  for (int64_t i = 0; i < n_values; i++) {
    for (int32_t k = 0; k < bpv; k++) {
      uint8_t hi = sym[t++], lo = sym[t++];
      if (hi > 15 || lo > 15) return -1;
      int32_t mem = msb_first ? (bpv - 1 - k) : k;
      values[i * bpv + mem] = (uint8_t)((hi << 4) | lo);
      byte_no++;
      if (bpg > 0 && (byte_no % bpg == 0 || byte_no == nbytes)) {
        if (sym[t++] != 16) return -1;
        if (nsep == 2 && sym[t++] != 17) return -1;
      }
    }
  }
  return 0;
}

/*
 * Brute-force check used by the tests: serialise and deserialise every 32-bit
 * pattern in [lo, hi) (as float32 values, 8 digits + separator) and compare.
 * Returns the number of mismatching patterns.
 */
int64_t orc_hex_roundtrip_range(uint64_t lo, uint64_t hi, int32_t msb_first) {
  enum { BLK = 4096 };
  static const int32_t ids[16] = {48, 49, 50, 51, 52, 53, 54, 55,
                                  56, 57, 97, 98, 99, 100, 101, 102};
  uint32_t* in = (uint32_t*)malloc(BLK * 4);
  uint32_t* out = (uint32_t*)malloc(BLK * 4);
  int32_t* tok = (int32_t*)malloc(BLK * 9 * sizeof(int32_t));
  uint8_t* sym = (uint8_t*)malloc(BLK * 9);
  int64_t bad = 0;
  for (uint64_t base = lo; base < hi; base += BLK) {
    int64_t n = (int64_t)((hi - base) < BLK ? (hi - base) : BLK);
    for (int64_t i = 0; i < n; i++) in[i] = (uint32_t)(base + i);
    int64_t nt = orc_serialize((const uint8_t*)in, n, 4, 4, msb_first, ids, 32, -1, tok, sym);
    for (int64_t t = 0; t < nt; t++) {
      int s = sym[t];
      int want = s < 16 ? ids[s] : 32;
      if (tok[t] != want) bad++;
    }
    if (orc_deserialize(sym, nt, n, 4, 4, msb_first, 1, (uint8_t*)out) != 0) {
      bad += n;
      continue;
    }
    for (int64_t i = 0; i < n; i++) bad += (in[i] != out[i]);
  }
  free(in); free(out); free(tok); free(sym);
  return bad;
}

/* ------------------------------------------------------------------------ */
/* Probability table                                                          */
/* ------------------------------------------------------------------------ */

/*
 * lp[na]: float32 natural-log probabilities of the na alphabet symbols (16
 * digits and the separator token(s)); escape bin na takes the rest, or
 * nothing when renorm is set (lp then sums to one over the alphabet).
 * cdf[na+2]: cdf[0] = 0, cdf[k+1] = cdf[k] + f_k, cdf[na+1] = total.
 */
void orc_quantize(const float* lp, int32_t na, int32_t renorm, uint32_t total, uint32_t* cdf) {
  int64_t f[ORC_NSYM_MAX];
  const int32_t nsym = na + 1;
  const uint32_t spread = renorm ? total - (uint32_t)na : total - (uint32_t)nsym;
  const int64_t alpha_total = renorm ? (int64_t)total : (int64_t)total - 1;
  int64_t s = 0;
  for (int a = 0; a < na; a++) {
    double p = exp((double)lp[a]);
    double q = floor(p * (double)spread);
    f[a] = 1 + (int64_t)q;
    s += f[a];
  }
  if (s > alpha_total || (renorm && s < alpha_total)) {
    int big = 0;
    for (int a = 1; a < na; a++)
      if (f[a] > f[big]) big = a;
    f[big] += alpha_total - s;
    s = alpha_total;
  }
  f[na] = (int64_t)total - s;
  cdf[0] = 0;
  for (int k = 0; k < nsym; k++) cdf[k + 1] = cdf[k] + (uint32_t)f[k];
}

void orc_quantize_rows(const float* lp, int64_t rows, int32_t na, int32_t renorm, uint32_t total,
                       uint32_t* cdf) {
  for (int64_t r = 0; r < rows; r++)
    orc_quantize(lp + r * na, na, renorm, total, cdf + r * (na + 2));
}

/* ------------------------------------------------------------------------ */
/* Arithmetic coder (Witten, Neal & Cleary 1987), 62-bit code values          */
/* ------------------------------------------------------------------------ */

#define CODE_BITS 62
#define TOP ((((uint64_t)1) << CODE_BITS) - 1)
#define HALF (((uint64_t)1) << (CODE_BITS - 1))
#define QUARTER (((uint64_t)1) << (CODE_BITS - 2))
#define THREE_Q (HALF + QUARTER)

typedef struct {
  uint8_t* out;
  uint64_t cap_bits;
  uint64_t nbits;
  int overflow;
} bitwriter;

static void put_bit(bitwriter* w, int bit) {
  if (w->nbits >= w->cap_bits) { w->overflow = 1; return; }
  uint64_t byte = w->nbits >> 3;
  int shift = 7 - (int)(w->nbits & 7);
  if (shift == 7) w->out[byte] = 0;
  if (bit) w->out[byte] |= (uint8_t)(1u << shift);
  w->nbits++;
}

static void put_bit_plus_pending(bitwriter* w, int bit, uint64_t* pending) {
  put_bit(w, bit);
  for (; *pending > 0; (*pending)--) put_bit(w, !bit);
}

/*
 * Encode n symbols; row j of cdf (nsym+1 entries, cdf[nsym] = total) is the
 * model for symbol j.  Writes whole bytes into out (cap bytes available).
 * Returns the number of bits, or -1 if out is too small, -2 on a bad symbol
 * (zero-frequency bin or out of range).
 */
int64_t orc_ac_encode(const uint32_t* cdf, int32_t nsym, const uint8_t* sym,
                      int64_t n, uint8_t* out, uint64_t cap) {
  bitwriter w = {out, cap * 8, 0, 0};
  uint64_t low = 0, high = TOP, pending = 0;
  for (int64_t j = 0; j < n; j++) {
    const uint32_t* c = cdf + j * (int64_t)(nsym + 1);
    int s = sym[j];
    if (s >= nsym || c[s + 1] <= c[s]) return -2;
    unsigned __int128 range = (unsigned __int128)(high - low) + 1;
    uint64_t total = c[nsym];
    high = low + (uint64_t)((range * c[s + 1]) / total) - 1;
    low = low + (uint64_t)((range * c[s]) / total);
    for (;;) {
      if (high < HALF) {
        put_bit_plus_pending(&w, 0, &pending);
      } else if (low >= HALF) {
        put_bit_plus_pending(&w, 1, &pending);
        low -= HALF;
        high -= HALF;
      } else if (low >= QUARTER && high < THREE_Q) {
        pending++;
        low -= QUARTER;
        high -= QUARTER;
      } else {
        break;
      }
      low = low << 1;
      high = (high << 1) | 1;
    }
  }
  pending++;
  if (low < QUARTER) put_bit_plus_pending(&w, 0, &pending);
  else put_bit_plus_pending(&w, 1, &pending);
  if (w.overflow) return -1;
  return (int64_t)w.nbits;
}

typedef struct {
  const uint8_t* in;
  uint64_t nbits;
  uint64_t pos;
  uint64_t low, high, value;
} orc_decoder;

static int get_bit(orc_decoder* d) {
  int bit = 0;
  if (d->pos < d->nbits) bit = (d->in[d->pos >> 3] >> (7 - (d->pos & 7))) & 1;
  d->pos++;
  return bit;
}

size_t orc_decoder_size(void) { return sizeof(orc_decoder); }

void orc_ac_decode_init(orc_decoder* d, const uint8_t* in, uint64_t nbits) {
  d->in = in;
  d->nbits = nbits;
  d->pos = 0;
  d->low = 0;
  d->high = TOP;
  d->value = 0;
  for (int i = 0; i < CODE_BITS; i++) d->value = (d->value << 1) | (uint64_t)get_bit(d);
}

/* Decode one symbol with model row c (nsym+1 entries).  Returns the symbol. */
int orc_ac_decode_symbol(orc_decoder* d, const uint32_t* c, int32_t nsym) {
  unsigned __int128 range = (unsigned __int128)(d->high - d->low) + 1;
  uint64_t total = c[nsym];
  /* largest cumulative count not above the scaled code value */
  uint64_t target = (uint64_t)((((unsigned __int128)(d->value - d->low) + 1) * total - 1) / range);
  int s = 0;
  while (s + 1 < nsym && c[s + 1] <= target) s++;
  d->high = d->low + (uint64_t)((range * c[s + 1]) / total) - 1;
  d->low = d->low + (uint64_t)((range * c[s]) / total);
  for (;;) {
    if (d->high < HALF) {
      /* nothing */
    } else if (d->low >= HALF) {
      d->value -= HALF;
      d->low -= HALF;
      d->high -= HALF;
    } else if (d->low >= QUARTER && d->high < THREE_Q) {
      d->value -= QUARTER;
      d->low -= QUARTER;
      d->high -= QUARTER;
    } else {
      break;
    }
    d->low = d->low << 1;
    d->high = (d->high << 1) | 1;
    d->value = (d->value << 1) | (uint64_t)get_bit(d);
  }
  return s;
}

/* Decode n symbols with a fixed sequence of model rows. */
void orc_ac_decode(const uint32_t* cdf, int32_t nsym, int64_t n, const uint8_t* in,
                   uint64_t nbits, uint8_t* sym) {
  orc_decoder d;
  orc_ac_decode_init(&d, in, nbits);
  for (int64_t j = 0; j < n; j++)
    sym[j] = (uint8_t)orc_ac_decode_symbol(&d, cdf + j * (int64_t)(nsym + 1), nsym);
}
