// Host side of the LM-GC boundary: arithmetic coding of windows against the
// per-position tables the LM produces (Sec. 3, "Arithmetic coding"; Sec. 4,
// "Compression"), the inverse of serialisation, and the container format.
//
// The coder is the Witten-Neal-Cleary binary arithmetic coder with 62-bit
// code values (128-bit products for the interval update), E1/E2/E3
// renormalisation with pending bits, and a flush of pending+1 bits whose
// first bit is 0 when low < 1/4.  Output bits are buffered 64 at a time.
// Windows are independent bitstreams and are coded on several host threads.
#include <string.h>

#include <algorithm>
#include <atomic>
#include <system_error>
#include <thread>
#include <vector>

#include "host.h"

namespace lmgc {
namespace {

constexpr int kCodeBits = 62;
constexpr uint64_t kTop = (uint64_t(1) << kCodeBits) - 1;
constexpr uint64_t kHalf = uint64_t(1) << (kCodeBits - 1);
constexpr uint64_t kQuarter = uint64_t(1) << (kCodeBits - 2);
constexpr uint64_t kThreeQuarters = kHalf + kQuarter;

typedef unsigned __int128 u128;

// MSB-first bit sink into a caller buffer.
class BitSink {
 public:
  BitSink(uint8_t* out, size_t cap) : out_(out), cap_(cap) {}
  void put(unsigned bit) {
    acc_ = (acc_ << 1) | bit;
    if (++nacc_ == 64) flush_word();
  }
  void put_repeat(unsigned bit, uint64_t n) {
    while (n--) put(bit);
  }
  // Pads the last byte with zero bits; returns false on overflow.
  bool finish() {
    if (nacc_ == 0) return !overflow_;
    const int full = nacc_ / 8, rem = nacc_ % 8;
    uint64_t a = acc_ << (64 - nacc_);  // left-align
    for (int i = 0; i < full + (rem ? 1 : 0); i++) emit_byte((uint8_t)(a >> (56 - 8 * i)));
    nacc_ = 0;
    acc_ = 0;
    return !overflow_;
  }
  uint64_t bits() const { return bits_base_ + nacc_; }
  size_t bytes() const { return pos_; }

 private:
  void flush_word() {
    for (int i = 0; i < 8; i++) emit_byte((uint8_t)(acc_ >> (56 - 8 * i)));
    acc_ = 0;
    nacc_ = 0;
    bits_base_ += 64;
  }
  void emit_byte(uint8_t b) {
    if (pos_ < cap_) out_[pos_] = b;
    else overflow_ = true;
    pos_++;
  }
  uint8_t* out_;
  size_t cap_;
  size_t pos_ = 0;
  uint64_t acc_ = 0;
  int nacc_ = 0;
  uint64_t bits_base_ = 0;
  bool overflow_ = false;
};

// Encodes one window.  Returns bits (>= 0), -1 overflow, -2 bad symbol.
int64_t encode_window(const uint32_t* cdf, int nsym, const uint8_t* sym, int n, uint8_t* out,
                      size_t cap) {
  BitSink sink(out, cap);
  uint64_t low = 0, high = kTop, pending = 0;
  const int stride = nsym + 1;
  for (int j = 0; j < n; j++) {
    const uint32_t* c = cdf + (size_t)j * stride;
    const unsigned s = sym[j];
    if (s >= (unsigned)nsym) return -2;
    const uint64_t lo_c = c[s], hi_c = c[s + 1], total = c[nsym];
    if (hi_c <= lo_c || hi_c > total) return -2;
    const u128 range = (u128)(high - low) + 1;
    high = low + (uint64_t)((range * hi_c) / total) - 1;
    low = low + (uint64_t)((range * lo_c) / total);
    for (;;) {
      if (high < kHalf) {
        sink.put(0);
        sink.put_repeat(1, pending);
        pending = 0;
      } else if (low >= kHalf) {
        sink.put(1);
        sink.put_repeat(0, pending);
        pending = 0;
        low -= kHalf;
        high -= kHalf;
      } else if (low >= kQuarter && high < kThreeQuarters) {
        pending++;
        low -= kQuarter;
        high -= kQuarter;
      } else {
        break;
      }
      low <<= 1;
      high = (high << 1) | 1;
    }
  }
  pending++;
  const unsigned first = low < kQuarter ? 0u : 1u;
  sink.put(first);
  sink.put_repeat(first ^ 1u, pending);
  const uint64_t bits = sink.bits();
  if (!sink.finish()) return -1;
  return (int64_t)bits;
}

struct DecState {
  const uint8_t* in;
  uint64_t nbits, pos, low, high, value;
};
static_assert(sizeof(DecState) <= sizeof(lmgc_decoder), "decoder state too large");

inline unsigned next_bit(DecState* d) {
  unsigned b = 0;
  if (d->pos < d->nbits) b = (d->in[d->pos >> 3] >> (7 - (d->pos & 7))) & 1u;
  d->pos++;
  return b;
}

}  // namespace

// --------------------------------------------------------------- encoding
int encode_windows(const uint32_t* cdf, int nsym, const uint8_t* sym, const int32_t* len,
                   int n_win, int W, uint8_t* out, size_t cap, uint32_t* bits, size_t* used,
                   int n_threads) {
  if (n_win <= 0) {
    *used = 0;
    return LMGC_OK;
  }
  const size_t bound = encode_bound_bytes(W);
  std::vector<uint8_t> scratch((size_t)n_win * bound);
  std::vector<int64_t> nb(n_win, 0);
  std::atomic<int> next(0);
  std::atomic<int> err(0);
  auto worker = [&]() {
    for (;;) {
      const int w = next.fetch_add(1);
      if (w >= n_win) break;
      const size_t off = (size_t)w * W;
      const int n = len[w];
      if (n < 0 || n > W) {
        err = LMGC_EINVAL;
        continue;
      }
      const int64_t b = encode_window(cdf + off * (nsym + 1), nsym, sym + off, n,
                                      scratch.data() + (size_t)w * bound, bound);
      if (b < 0) err = (b == -2) ? LMGC_ECORRUPT : LMGC_ESIZE;
      nb[w] = b;
    }
  };
  int T = n_threads > 0 ? n_threads : (int)std::min(8u, std::max(1u, std::thread::hardware_concurrency()));
  T = std::min(T, n_win);
  std::vector<std::thread> pool;
  pool.reserve(T);  // no reallocation below, so only a thread start can fail
  for (int t = 1; t < T; t++) {
    try {
      pool.emplace_back(worker);
    } catch (const std::system_error&) {
      break;  // run with the threads that did start
    }
  }
  worker();
  for (auto& th : pool) th.join();
  if (err.load()) {
    return set_error(err.load(), err.load() == LMGC_ECORRUPT
                                     ? "lmgc_encode: symbol with zero frequency or out of range"
                                     : "lmgc_encode: invalid window length");
  }
  size_t pos = 0;
  for (int w = 0; w < n_win; w++) {
    const size_t bytes = (size_t)(nb[w] + 7) / 8;
    if (pos + bytes > cap) return set_error(LMGC_ESIZE, "lmgc_encode: output buffer too small");
    memcpy(out + pos, scratch.data() + (size_t)w * bound, bytes);
    bits[w] = (uint32_t)nb[w];
    pos += bytes;
  }
  *used = pos;
  return LMGC_OK;
}

size_t encode_bound_bytes(int W) {
  // each symbol narrows the interval by at least 1/T <= 2^-32: <= 33 bits,
  // plus the flush
  return ((size_t)W * 33 + 64 + 7) / 8 + 8;
}

// --------------------------------------------------------------- decoding
int decoder_init(lmgc_decoder* st, const uint8_t* payload, uint64_t nbits) {
  DecState* d = reinterpret_cast<DecState*>(st);
  d->in = payload;
  d->nbits = nbits;
  d->pos = 0;
  d->low = 0;
  d->high = kTop;
  d->value = 0;
  for (int i = 0; i < kCodeBits; i++) d->value = (d->value << 1) | next_bit(d);
  return LMGC_OK;
}

int decoder_symbol(lmgc_decoder* st, const uint32_t* c, int nsym, int32_t* out) {
  DecState* d = reinterpret_cast<DecState*>(st);
  const uint64_t total = c[nsym];
  if (total == 0 || d->value < d->low || d->value > d->high)
    return set_error(LMGC_ECORRUPT, "lmgc_decode_symbol: inconsistent state");
  const u128 range = (u128)(d->high - d->low) + 1;
  const uint64_t target = (uint64_t)((((u128)(d->value - d->low) + 1) * total - 1) / range);
  // binary search: largest s with c[s] <= target
  int lo = 0, hi = nsym;  // c[lo] <= target < c[hi]
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (c[mid] <= target) lo = mid;
    else hi = mid;
  }
  const int s = lo;
  d->high = d->low + (uint64_t)((range * c[s + 1]) / total) - 1;
  d->low = d->low + (uint64_t)((range * c[s]) / total);
  for (;;) {
    if (d->high < kHalf) {
    } else if (d->low >= kHalf) {
      d->value -= kHalf;
      d->low -= kHalf;
      d->high -= kHalf;
    } else if (d->low >= kQuarter && d->high < kThreeQuarters) {
      d->value -= kQuarter;
      d->low -= kQuarter;
      d->high -= kQuarter;
    } else {
      break;
    }
    d->low <<= 1;
    d->high = (d->high << 1) | 1;
    d->value = (d->value << 1) | next_bit(d);
  }
  *out = s;
  return LMGC_OK;
}

// ---------------------------------------------------------- serialisation
int64_t num_tokens(int64_t n_values, const lmgc_serial_params& p) {
  if (n_values < 0 || n_values > LMGC_MAX_VALUES) return -1;
  const int64_t nbytes = n_values * p.bytes_per_value;
  const int64_t groups = p.bytes_per_group > 0 ? (nbytes + p.bytes_per_group - 1) / p.bytes_per_group : 0;
  return 2 * nbytes + groups * (p.sep2_id >= 0 ? 2 : 1);
}

int deserialize_bins(const uint8_t* sym, int64_t n_tokens, int64_t n_values,
                     const lmgc_serial_params& p, uint8_t* out) {
  if (num_tokens(n_values, p) != n_tokens)
    return set_error(LMGC_ECORRUPT, "lmgc_deserialize: token count does not match value count");
  const int bpv = p.bytes_per_value, bpg = p.bytes_per_group;
  const int64_t nbytes = n_values * bpv;
  int64_t t = 0;
  int in_group = 0;
  for (int64_t byte = 0; byte < nbytes; byte++) {
    const unsigned hi = sym[t], lo = sym[t + 1];
    t += 2;
    if (hi > 15 || lo > 15) return set_error(LMGC_ECORRUPT, "lmgc_deserialize: digit expected");
    const int64_t v = byte / bpv;
    const int k = (int)(byte - v * bpv);
    out[v * bpv + (p.msb_first ? bpv - 1 - k : k)] = (uint8_t)((hi << 4) | lo);
    if (bpg > 0 && (++in_group == bpg || byte + 1 == nbytes)) {
      in_group = 0;
      if (sym[t++] != 16) return set_error(LMGC_ECORRUPT, "lmgc_deserialize: separator expected");
      if (p.sep2_id >= 0 && sym[t++] != 17) return set_error(LMGC_ECORRUPT, "lmgc_deserialize: separator expected");
    }
  }
  return LMGC_OK;
}

// --------------------------------------------------------------- container
static void put_u16(uint8_t* p, uint16_t v) { memcpy(p, &v, 2); }
static void put_u32(uint8_t* p, uint32_t v) { memcpy(p, &v, 4); }
static void put_u64(uint8_t* p, uint64_t v) { memcpy(p, &v, 8); }
static uint16_t get_u16(const uint8_t* p) { uint16_t v; memcpy(&v, p, 2); return v; }
static uint32_t get_u32(const uint8_t* p) { uint32_t v; memcpy(&v, p, 4); return v; }
static uint64_t get_u64(const uint8_t* p) { uint64_t v; memcpy(&v, p, 8); return v; }

void write_header(uint8_t* h, const ContainerHeader& c) {
  memset(h, 0, LMGC_HEADER_BYTES);
  memcpy(h, "LMGC", 4);
  put_u16(h + 4, 1);
  put_u16(h + 6, LMGC_HEADER_BYTES);
  put_u64(h + 8, c.model_tag);
  put_u64(h + 16, (uint64_t)c.n_values);
  h[24] = (uint8_t)c.p.bytes_per_value;
  h[25] = (uint8_t)c.p.bytes_per_group;
  h[26] = (uint8_t)c.p.msb_first;
  h[27] = (uint8_t)(c.p.sep2_id >= 0 ? LMGC_NALPHA_MAX + 1 : LMGC_NALPHA + 1);
  put_u32(h + 28, (uint32_t)c.p.window);
  put_u32(h + 32, c.total);
  put_u32(h + 36, (uint32_t)c.n_windows);
  put_u32(h + 40, (uint32_t)c.p.bos_id);
  put_u32(h + 44, (uint32_t)c.p.pad_id);
  put_u32(h + 48, (uint32_t)c.p.sep_id);
  for (int i = 0; i < 16; i++) put_u32(h + 52 + 4 * i, (uint32_t)c.p.hex_ids[i]);
  put_u32(h + 116, (uint32_t)(c.p.sep2_id + 1));
  put_u32(h + 120, (uint32_t)c.p.renorm);
}

int read_header(const uint8_t* buf, size_t bytes, ContainerHeader* c) {
  if (bytes < LMGC_HEADER_BYTES || memcmp(buf, "LMGC", 4) != 0)
    return set_error(LMGC_ECORRUPT, "container: bad magic or truncated header");
  if (get_u16(buf + 4) != 1 || get_u16(buf + 6) != LMGC_HEADER_BYTES)
    return set_error(LMGC_ECORRUPT, "container: unsupported version");
  c->model_tag = get_u64(buf + 8);
  c->n_values = (int64_t)get_u64(buf + 16);
  c->p.bytes_per_value = buf[24];
  c->p.bytes_per_group = buf[25];
  c->p.msb_first = buf[26];
  c->p.window = (int32_t)get_u32(buf + 28);
  c->total = get_u32(buf + 32);
  c->n_windows = get_u32(buf + 36);
  c->p.bos_id = (int32_t)get_u32(buf + 40);
  c->p.pad_id = (int32_t)get_u32(buf + 44);
  c->p.sep_id = (int32_t)get_u32(buf + 48);
  for (int i = 0; i < 16; i++) c->p.hex_ids[i] = (int32_t)get_u32(buf + 52 + 4 * i);
  c->p.sep2_id = (int32_t)(get_u32(buf + 116) - 1u);  // 0 (none) -> -1
  c->p.renorm = (int32_t)get_u32(buf + 120);
  if (c->p.renorm != 0 && c->p.renorm != 1) return set_error(LMGC_ECORRUPT, "container: bad table mode");
  if (buf[27] != (c->p.sep2_id >= 0 ? LMGC_NALPHA_MAX + 1 : LMGC_NALPHA + 1))
    return set_error(LMGC_ECORRUPT, "container: symbol count does not match the separators");
  if (c->n_values < 0 || c->n_values > LMGC_MAX_VALUES || c->p.window <= 0 ||
      (c->p.bytes_per_value != 1 && c->p.bytes_per_value != 2 && c->p.bytes_per_value != 4))
    return set_error(LMGC_ECORRUPT, "container: bad header fields");
  const int64_t nt = num_tokens(c->n_values, c->p);
  if ((nt + c->p.window - 1) / c->p.window != c->n_windows)
    return set_error(LMGC_ECORRUPT, "container: window count does not match the vector size");
  if (bytes < LMGC_HEADER_BYTES + 4 * (size_t)c->n_windows)
    return set_error(LMGC_ECORRUPT, "container: truncated bit-count table");
  return LMGC_OK;
}

}  // namespace lmgc
