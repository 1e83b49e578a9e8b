// Host-side internal declarations of liblmgc (errors, coder, container).
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/lmgc.h"

namespace lmgc {

// Records a thread-local error message and returns `code`.
int set_error(int code, const char* fmt, ...);
void clear_error();

// ---- arithmetic coder
size_t encode_bound_bytes(int W);
int encode_windows(const uint32_t* cdf, int nsym, const uint8_t* sym, const int32_t* len,
                   int n_win, int W, uint8_t* out, size_t cap, uint32_t* bits, size_t* used,
                   int n_threads);
int decoder_init(lmgc_decoder* st, const uint8_t* payload, uint64_t nbits);
int decoder_symbol(lmgc_decoder* st, const uint32_t* cdf_row, int nsym, int32_t* out);

// ---- serialisation
int64_t num_tokens(int64_t n_values, const lmgc_serial_params& p);
int deserialize_bins(const uint8_t* sym, int64_t n_tokens, int64_t n_values,
                     const lmgc_serial_params& p, uint8_t* out);

// ---- container
struct ContainerHeader {
  uint64_t model_tag;
  int64_t n_values;
  lmgc_serial_params p;
  uint32_t total;
  int64_t n_windows;
};
void write_header(uint8_t* h, const ContainerHeader& c);
int read_header(const uint8_t* buf, size_t bytes, ContainerHeader* c);

}  // namespace lmgc
