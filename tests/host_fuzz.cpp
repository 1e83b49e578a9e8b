// Randomised check of the host coder, container header parser and
// deserialiser, built with AddressSanitizer and UndefinedBehaviorSanitizer
// by tests/test_host_fuzz.py: encode -> decode round trips on random tables
// (some streams corrupted: those must not crash), mutated headers, random bins.
// Error reporting is stubbed; the library records messages per thread.
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>
#include <random>
#include <vector>
#include "../paper_2409_17836_amd/csrc/host.h"
namespace lmgc {
int set_error(int code, const char* fmt, ...) { return code; }
void clear_error() {}
}
using namespace lmgc;
int main(int argc, char** argv) {
  std::mt19937_64 rng(argc > 1 ? atoi(argv[1]) : 1);
  long ok = 0, errs = 0, mism = 0;
  for (int it = 0; it < 3000; it++) {
    const int nsym = 18 + (rng() % 2), W = 1 + rng() % 300, nwin = 1 + rng() % 5;
    const uint32_t T = (rng() % 2) ? (1u << 16) : (1u << 24);
    std::vector<uint32_t> cdf((size_t)nwin * W * (nsym + 1));
    std::vector<uint8_t> sym((size_t)nwin * W);
    std::vector<int32_t> len(nwin);
    for (int w = 0; w < nwin; w++) len[w] = rng() % (W + 1);
    for (size_t r = 0; r < (size_t)nwin * W; r++) {
      uint32_t* c = &cdf[r * (nsym + 1)];
      std::vector<uint32_t> f(nsym);
      uint32_t s = 0;
      for (int k = 0; k < nsym; k++) { f[k] = 1 + (rng() % 4 == 0 ? rng() % (T / nsym) : rng() % 8); s += f[k]; }
      if (s > T) { for (int k = 0; k < nsym; k++) f[k] = 1; s = nsym; }
      f[rng() % nsym] += T - s;
      c[0] = 0;
      for (int k = 0; k < nsym; k++) c[k + 1] = c[k] + f[k];
      uint32_t pick;
      do { pick = rng() % nsym; } while (f[pick] == 0);
      sym[r] = (uint8_t)pick;
    }
    std::vector<uint8_t> out(nwin * encode_bound_bytes(W) + 16);
    std::vector<uint32_t> bits(nwin);
    size_t used = 0;
    int rc = encode_windows(cdf.data(), nsym, sym.data(), len.data(), nwin, W, out.data(), out.size(), bits.data(), &used, 1 + rng() % 3);
    if (rc) { errs++; continue; }
    size_t off = 0;
    for (int w = 0; w < nwin; w++) {
      const size_t nb = (bits[w] + 7) / 8;
      std::vector<uint8_t> pay(out.begin() + off, out.begin() + off + nb);
      // corrupt some streams: flip bytes, truncate the bit count
      uint64_t nbits = bits[w];
      const bool bad = rng() % 3 == 0;
      if (bad && nb) { pay[rng() % nb] ^= 1 + rng() % 255; if (rng() % 2) nbits = rng() % (nbits + 1); }
      lmgc_decoder st;
      if (decoder_init(&st, pay.data(), nbits)) { errs++; off += nb; continue; }
      for (int j = 0; j < len[w]; j++) {
        int32_t s = -1;
        if (decoder_symbol(&st, &cdf[((size_t)w * W + j) * (nsym + 1)], nsym, &s)) { errs++; break; }
        if (s < 0 || s >= nsym) { printf("symbol out of range\n"); return 1; }
        if (!bad && s != sym[(size_t)w * W + j]) { mism++; break; }
      }
      off += nb;
      ok++;
    }
    if (off != used) { printf("size mismatch\n"); return 1; }
    // header parser on a valid header and on mutations
    uint8_t h[LMGC_HEADER_BYTES + 64];
    ContainerHeader c = {};
    c.model_tag = rng(); c.n_values = rng() % 100000; c.p.bytes_per_value = 4; c.p.bytes_per_group = 4;
    c.p.msb_first = 1; c.p.window = 1 + rng() % 5000; c.p.bos_id = 1; c.p.pad_id = 1; c.p.sep_id = 32;
    for (int i = 0; i < 16; i++) c.p.hex_ids[i] = i < 10 ? 48 + i : 87 + i;
    c.p.sep2_id = -1; c.p.renorm = 0; c.total = 1 << 16;
    c.n_windows = (num_tokens(c.n_values, c.p) + c.p.window - 1) / c.p.window;
    write_header(h, c);
    ContainerHeader r;
    const size_t hb = LMGC_HEADER_BYTES + 4 * (size_t)c.n_windows;
    std::vector<uint8_t> full(hb + 8, 0);
    memcpy(full.data(), h, LMGC_HEADER_BYTES);
    if (read_header(full.data(), full.size(), &r)) { printf("valid header rejected\n"); return 1; }
    for (int m = 0; m < 20; m++) {
      std::vector<uint8_t> mut = full;
      mut[rng() % LMGC_HEADER_BYTES] = (uint8_t)rng();
      read_header(mut.data(), rng() % (mut.size() + 1), &r);
    }
    // deserialiser on random bins
    const int64_t nv = rng() % 50;
    lmgc_serial_params p = c.p;
    p.bytes_per_group = rng() % 9;
    const int64_t nt = num_tokens(nv, p);
    std::vector<uint8_t> bins(nt + 1);
    for (auto& b : bins) b = rng() % 18;
    std::vector<uint8_t> vals(nv * 4 + 1);
    deserialize_bins(bins.data(), nt, nv, p, vals.data());
  }
  printf("ok %ld errs %ld mismatches %ld\n", ok, errs, mism);
  return mism ? 1 : 0;
}
