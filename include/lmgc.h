/*
 * lmgc.h -- C ABI of liblmgc, an MI355X (gfx950) implementation of the LM-GC
 * hot path: "Language Models as Zero-shot Lossless Gradient Compressors"
 * (arXiv 2409.17836).
 *
 * The method (Sec. 4): serialise float32 gradients as hexadecimal text with a
 * separator after every 4 bytes, run a causal language model over the token
 * stream to get p(t_k | BOS, t_<k) for every token (Eq. 2), and use these
 * probabilities as the model of an arithmetic coder (Sec. 3, "Arithmetic
 * coding"); decompression replays the model from BOS token by token.
 *
 * Conventions
 *   - Every call returns an int status (LMGC_OK or a negative LMGC_E* code)
 *     unless stated otherwise; lmgc_last_error() gives a thread-local message.
 *     No C++ exception or abort crosses this ABI: a failed host allocation
 *     returns LMGC_ENOMEM.
 *   - The caller owns every buffer.  "d_" pointers are device (HBM) pointers,
 *     "h_"/plain pointers are host pointers.  Size helpers say how much to
 *     allocate.
 *   - GPU calls are asynchronous on the caller's stream (a hipStream_t passed
 *     as void*; NULL = the default stream).  Host calls are synchronous.
 *   - Layouts are row-major, little-endian.
 *   - A model handle is immutable after lmgc_model_create and may be used
 *     from several host threads with different workspaces.
 */
#ifndef LMGC_H
#define LMGC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ----------------------------------------------------------------- status */
#define LMGC_OK 0
#define LMGC_EINVAL -1        /* bad argument or unsupported shape          */
#define LMGC_ENOMEM -2        /* device or host allocation failed           */
#define LMGC_EDEVICE -3       /* a HIP runtime call failed                  */
#define LMGC_ESIZE -4         /* caller buffer too small                    */
#define LMGC_ECORRUPT -5      /* malformed token stream, bitstream or container */
#define LMGC_EUNSUPPORTED -6  /* valid request this build does not support  */

/* Thread-local description of the last error on this thread ("" if none). */
const char* lmgc_last_error(void);

/* Library version string. */
const char* lmgc_version(void);

/* ---------------------------------------------------------- serialisation */
/*
 * Serialisation parameters (Sec. 4, "Serialization"; byte-grouping ablation
 * in Sec. 5.3).  The value vector is read as a stream of bytes, each value's
 * bytes most-significant first when msb_first=1 (sign/exponent digits lead,
 * like printf("%08x")) or in memory (little-endian) order when msb_first=0;
 * each byte gives two hex-digit tokens, high nibble first; the separator
 * (sep_id, then sep2_id if >= 0) follows every bytes_per_group bytes and the
 * last (possibly partial) group.  bytes_per_group = 0 means no separator (the
 * paper's H_n).  The paper's separators (Sec. 5.2, Table 1) are one space
 * (H_s), a comma (H_c), a semicolon (H_semi) or a comma and a space (H_c+s:
 * sep_id = ',' and sep2_id = ' ').  With bytes_per_value = bytes_per_group =
 * 4 every float32 is 8 digits + 1 separator = 9 tokens (10 with sep2_id).
 *
 * The stream is cut into consecutive windows of `window` tokens (the last
 * one shorter; its tail is filled with pad_id).  The model input of a window
 * is BOS followed by the window's tokens shifted by one, so position j is
 * predicted from BOS and tokens 0..j-1 (Eq. 2); BOS is never coded.
 *
 * Coder bins: 0..15 = hex digit value, 16 = sep_id, then 17 = sep2_id when
 * there is one, then the escape bin (the rest of the vocabulary; never
 * coded).  The alphabet (bins before the escape) has A = 17 or 18 symbols
 * (lmgc_alphabet_size); tables have A + 2 entries.  Alphabet ids must be
 * pairwise distinct and, like bos_id and pad_id, < the model's vocabulary.
 *
 * Tables (Sec. 4, the LM's distribution is the coder's model): with renorm =
 * 0 the alphabet bins carry the LM's probabilities over the whole vocabulary
 * and the escape bin the rest; with renorm = 1 the distribution is restricted
 * to the alphabet and renormalised over it (log-softmax over the A alphabet
 * logits; only those A columns of the LM head are evaluated), and the escape
 * bin is empty (cdf[A] = cdf[A+1] = total).
 */
typedef struct {
  int32_t bytes_per_value; /* 4 (float32) | 2 | 1 (8-bit indices) */
  int32_t bytes_per_group; /* >= 0 */
  int32_t msb_first;       /* 1 or 0 */
  int32_t window;          /* W > 0 */
  int32_t bos_id;
  int32_t pad_id;
  int32_t sep_id;
  int32_t hex_ids[16];
  int32_t sep2_id;         /* second separator token, or -1 (none) */
  int32_t renorm;          /* 0: full-vocabulary tables + escape; 1: renormalised */
} lmgc_serial_params;

#define LMGC_NALPHA 17     /* alphabet with one separator token        */
#define LMGC_NALPHA_MAX 18 /* alphabet with two separator tokens        */
#define LMGC_NSYM_MAX 19   /* coder bins incl. escape, at most          */

/* Alphabet size A (17 or 18) of these parameters, or < 0 if invalid. */
int32_t lmgc_alphabet_size(const lmgc_serial_params* p);

/* Largest vector the library takes (values): token counts stay far from
 * int64 overflow.  Larger counts are errors (EINVAL; ECORRUPT in a header). */
#define LMGC_MAX_VALUES (1LL << 56)

/* Tokens in the serialised stream of n_values values (0 <= n_values <=
 * LMGC_MAX_VALUES), or < 0 on error. */
int64_t lmgc_num_tokens(int64_t n_values, const lmgc_serial_params* p);
/* Windows the stream is cut into (ceil(tokens / W)), or < 0 on error. */
int64_t lmgc_num_windows(int64_t n_values, const lmgc_serial_params* p);

/*
 * Serialisation (Sec. 4, "Serialization"): windows [first_window,
 * first_window + n_windows) of the token stream of d_values (n_values values
 * of bytes_per_value bytes, device memory).  A range rather than the whole
 * stream, so that one batch of windows goes straight into the LM's input
 * buffer; the whole stream is first_window = 0, n_windows =
 * lmgc_num_windows(). d_tokens must be 16-byte and d_sym 4-byte aligned.
 *   d_tokens: [n_windows, W] int32 token ids; positions past the end of the
 *             stream get pad_id.
 *   d_sym:    nullable; [n_windows, W] uint8 coder bins (255 past the end).
 * GPU, async on stream.  Errors: EINVAL (bad params or window range).
 */
int lmgc_serialize(const void* d_values, int64_t n_values, const lmgc_serial_params* p,
                   int64_t first_window, int64_t n_windows, int32_t* d_tokens,
                   uint8_t* d_sym, void* stream);

/*
 * Host inverse of the serialisation (Sec. 4: decoding ends by mapping the
 * decoded text back to the float32 values) on coder bins: sym[n_tokens] ->
 * values_out (n_values * bytes_per_value bytes).  ECORRUPT if a digit or separator is out of place,
 * a bin is out of range or n_tokens does not match n_values.
 */
int lmgc_deserialize(const uint8_t* sym, int64_t n_tokens, int64_t n_values,
                     const lmgc_serial_params* p, void* values_out);

/* ------------------------------------------------------------ lossy steps */
/*
 * Lossy gradient compression that LM-GC is composed with (Sec. 5.4,
 * "Compatibility"): sparsification keeping a given share of the values,
 * linear quantisation to n-bit indices (Eq. 4), and one sign bit per value
 * (the 1-bit case, SignSGD).  Their outputs are value streams for
 * lmgc_serialize / lmgc_compress: float32 (bytes_per_value 4), uint8 indices
 * (1) and uint16 indices (2), packed sign bytes (1).
 *
 * Device pointers must be 16-byte aligned; n_values <= 2^31 - 1.
 */

/*
 * Number of values sparsification keeps when it keeps `percent` percent of
 * n_values values (Sec. 5.4 keeps 50, 25 and 10 percent):
 * floor(n_values * percent / 100).  Returns < 0 if n_values is outside
 * [0, 2^31 - 1] or percent outside [0, 100].  Host, pure arithmetic.
 */
int64_t lmgc_keep_count(int64_t n_values, int32_t percent);

/* Device workspace bytes of lmgc_sparsify_topk and lmgc_quantize_linear
 * (a few tens of KiB, independent of n_values), or < 0 if n_values is bad. */
int64_t lmgc_lossy_workspace(int64_t n_values);

/*
 * Sparsification (Sec. 5.4): keep the k values of largest magnitude, write
 * +0.0 in place of every other value; the stream keeps its length.
 * Magnitude is the IEEE bit pattern with the sign bit cleared, read as an
 * unsigned integer (the order of |v| for numbers, +0.0 and -0.0 equal, NaN
 * above infinity).  Ties are kept in index order (lower index first).
 *   d_values: float32 [n_values];  d_out: float32 [n_values], may equal
 *   d_values (in place) but must not overlap it otherwise.
 *   k: number kept, 0 <= k; k >= n_values keeps everything.  The paper's
 *   "keep p percent" is k = floor(n_values * p / 100).
 * GPU, async on stream (a chain of small launches: four histogram passes,
 * a tie count and one ordered write).  Errors: EINVAL, ESIZE (workspace).
 */
int lmgc_sparsify_topk(const float* d_values, int64_t n_values, int64_t k, float* d_out,
                       void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * lmgc_sparsify_topk without a workspace argument and without allocating,
 * for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc).  Same
 * arguments, result (bit for bit) and errors as lmgc_sparsify_topk, whose
 * kernels it runs.  The scratch is the library's own: a 32 KiB device array
 * that every GPU the library runs on holds until the process ends, found on
 * the caller's current device, which must be the device of the buffers and
 * the stream.  The call allocates nothing (no hipMalloc, no host staging).
 * Sizes: n_values in [0, 2^31 - 1], as for lmgc_sparsify_topk; the scratch
 * does not grow with n_values (EINVAL beyond that range).  Calls that
 * overlap on one GPU share the scratch and race: serialise them (one stream,
 * or events).  Errors: EINVAL, ESIZE, EDEVICE.
 */
int lmgc_sparsify_topk_noalloc(const float* d_values, int64_t n_values, int64_t k, float* d_out,
                               void* stream);

/*
 * Linear quantisation (Sec. 5.4, Eq. 4) of d_values to bits-bit indices:
 * idx = round-half-even(((v - min) / (max - min)) * (2^bits - 1)), each
 * operation in float32 with one rounding and no fused multiply-add; min and
 * max over the whole vector.  A constant vector gives all zeros.
 *   bits: 1..16.  d_indices: uint8 [n_values] for bits <= 8, uint16
 *   [n_values] for bits > 8.
 *   min_max: nullable host float[2]; receives (min, max), the values a
 *   receiver needs to map indices back.
 * Synchronises the stream once (min and max are read back to validate them)
 * and then enqueues the quantisation.  Errors: EINVAL (bad arguments, or the
 * vector holds a NaN or an infinity), ESIZE (workspace), EDEVICE.
 */
int lmgc_quantize_linear(const float* d_values, int64_t n_values, int32_t bits, void* d_indices,
                         float* min_max, void* d_workspace, size_t workspace_bytes, void* stream);

/*
 * One sign bit per value (Sec. 5.4, the 1-bit case read as SignSGD): the
 * IEEE sign bit (1 for negative numbers and -0.0), eight values per byte,
 * the first value in the most significant bit, the last byte padded with
 * zero bits.  d_out: uint8 [ceil(n_values / 8)].
 * GPU, async on stream.  Errors: EINVAL.
 */
int lmgc_sign_pack(const float* d_values, int64_t n_values, uint8_t* d_out, void* stream);

/* ------------------------------------------------------------------ model */
enum { LMGC_ARCH_LLAMA = 0, LMGC_ARCH_GPT2 = 1 };
enum { LMGC_DTYPE_F32 = 0, LMGC_DTYPE_BF16 = 1 };

/*
 * Decoder shape.  LLAMA: RMSNorm, RoPE (rotate-half, theta), SwiGLU FFN,
 * grouped-query attention (kv head of query head h = h*n_kv_heads/n_heads),
 * untied LM head.  GPT2: LayerNorm with bias, learned positions (max_pos),
 * biased projections, tanh-GELU FFN, head tied to the token embedding.
 * Requirements: d_model = n_heads * head_dim; head_dim in {64, 128} for BF16
 * and 16..64 (multiple of 16) for F32; d_model and d_ff multiples of 64.
 */
typedef struct {
  int32_t arch;       /* LMGC_ARCH_* */
  int32_t dtype;      /* LMGC_DTYPE_*: parameters and matrix-product operands */
  int32_t n_layers;
  int32_t d_model;
  int32_t n_heads;
  int32_t n_kv_heads;
  int32_t d_ff;
  int32_t vocab;
  int32_t max_pos;    /* longest window the model accepts */
  float rope_theta;
  float norm_eps;
} lmgc_model_config;

typedef struct lmgc_model lmgc_model;

/* Number of parameter tensors of a config, or < 0 on error. */
int32_t lmgc_model_num_tensors(const lmgc_model_config* cfg);

/*
 * Name (NUL-terminated, truncated to name_cap) and shape of manifest tensor
 * `index`.  Matrices are [out, in]: row n holds the weights of output
 * feature n.  LLAMA order: tok_emb[V,d]; per layer l: l{l}.attn_norm[d],
 * wq[Hq*hd,d], wk[Hkv*hd,d], wv[Hkv*hd,d], wo[d,Hq*hd], ffn_norm[d],
 * w_gate[F,d], w_up[F,d], w_down[d,F]; final_norm[d], lm_head[V,d].
 * GPT2 order: wte[V,d], wpe[max_pos,d]; per layer: ln1_g, ln1_b, w_qkv[3d,d],
 * b_qkv[3d], w_o[d,d], b_o[d], ln2_g, ln2_b, w_fc[F,d], b_fc[F],
 * w_proj[d,F], b_proj[d]; lnf_g[d], lnf_b[d].
 */
int lmgc_model_tensor_info(const lmgc_model_config* cfg, int32_t index, char* name,
                           size_t name_cap, int32_t* ndim, int64_t shape[2]);

/*
 * The LLM that serves as the prior (Sec. 5.1 uses pretrained TinyLlama,
 * OpenLLaMA and LLaMA-2; any weights of a supported shape work).  Create a
 * model from device tensors in manifest order, each of the config's dtype
 * (bfloat16 bit patterns for BF16); the caller loads them with any loader
 * (no weight file format is defined here).  The handle copies and repacks
 * what it needs into its own device memory (the caller may free the inputs
 * after the call returns).  Synchronises `stream`.
 * Errors: EINVAL (bad config), ENOMEM, EDEVICE.
 */
int lmgc_model_create(const lmgc_model_config* cfg, const void* const* d_weights,
                      void* stream, lmgc_model** out);
void lmgc_model_destroy(lmgc_model* m);

/* Bytes of device workspace lmgc_probs needs for B windows of W tokens. */
size_t lmgc_probs_workspace(const lmgc_model* m, int32_t B, int32_t W);

/*
 * The LM as the coder's model (Sec. 4, "Compression": P_AC = P_LM).
 * d_tokens: [B, W] int32 data tokens of B windows (the BOS shift is done
 * here).  With A = lmgc_alphabet_size(p), for every window b and position
 * j < W:
 *   lp[a]  = log p(alphabet token a | BOS, tokens[b, 0..j-1]), normalised
 *            over the whole vocabulary (float32, a = 0..A-1);
 *   f[a]   = 1 + floor(exp(lp[a]) * (total - (A+1))) (in double), the
 *            largest giving up any excess over total-1 (lowest index on ties);
 *   f[A]   = total - sum(f[0..A-1])  (escape bin, never coded);
 *   d_cdf[b, j, 0..A+1] = 0, f0, f0+f1, ..., total.
 * d_logp (nullable) receives lp as [B, W, A] float32.
 * Row (b, j) is a bitwise function of the weights and tokens[b, 0..j-1]
 * only: it does not depend on later tokens, on other windows, on B or on W.
 * total must be in [2*LMGC_NSYM_MAX, 2^24].  GPU, async.  Errors: EINVAL,
 * ESIZE (ws).
 */
int lmgc_probs(const lmgc_model* m, const int32_t* d_tokens, int32_t B, int32_t W,
               const lmgc_serial_params* p, uint32_t total, uint32_t* d_cdf, float* d_logp,
               void* d_ws, size_t ws_bytes, void* stream);

/*
 * The same tables as lmgc_probs, computed one position at a time the way the
 * decoder computes them (Sec. 4, "Compression": decompression starts from
 * BOS and feeds each decoded token back): every step runs the LM on one row
 * per window, reading the K and V of earlier positions from a per-layer
 * cache.  Each row's arithmetic is the one lmgc_probs does for that row, so
 * d_cdf (and d_logp) equal lmgc_probs' outputs bit for bit; tests use this
 * to check the decoder's path without arithmetic coding.  d_tokens [B, W]
 * device, B <= 32, other arguments and layouts as lmgc_probs.  Workspace:
 * lmgc_step_workspace(m, B, W) bytes (0 if B > 32).  GPU, async.
 */
size_t lmgc_step_workspace(const lmgc_model* m, int32_t B, int32_t W);
int lmgc_probs_stepwise(const lmgc_model* m, const int32_t* d_tokens, int32_t B, int32_t W,
                        const lmgc_serial_params* p, uint32_t total, uint32_t* d_cdf,
                        float* d_logp, void* d_ws, size_t ws_bytes, void* stream);

/* ---------------------------------------------------------------- coding */
/*
 * Arithmetic coding (Sec. 3): a Witten-Neal-Cleary binary arithmetic coder
 * with 62-bit code values.  Each window is an independent bitstream, packed
 * most significant bit first and padded with zero bits to a whole byte.
 * Flush: pending+1 bits, the first 0 if low < 1/4 else 1.
 */
/* Upper bound of the payload bytes lmgc_encode writes for these windows
 * (Sec. 3: at most 2 bits above the code length, per window). */
size_t lmgc_encode_bound(int32_t n_win, int32_t W);

/*
 * Arithmetic encoding of windows with the LM's tables (Sec. 3; Sec. 4,
 * "Compression").  Host.  cdf: [n_win, W, nsym+1] uint32 tables (cdf[..., nsym] = total);
 * sym: [n_win, W] bins; len[w] <= W symbols of window w are coded.
 * Writes the windows' payloads back to back into out (cap bytes); bits[w]
 * gets window w's exact bit count and *used the bytes written.
 * n_threads <= 0 picks a default.  Errors: EINVAL, ESIZE, ECORRUPT (a symbol
 * with zero frequency or out of range).
 */
int lmgc_encode(const uint32_t* cdf, int32_t nsym, const uint8_t* sym, const int32_t* len,
                int32_t n_win, int32_t W, uint8_t* out, size_t cap, uint32_t* bits,
                size_t* used, int32_t n_threads);

/* Symbol-at-a-time decoder state (opaque). */
typedef struct {
  uint64_t opaque[8];
} lmgc_decoder;

/* Arithmetic decoding (Sec. 3), one symbol at a time, so that the table of
 * the next position can be computed from the symbols decoded so far
 * (Sec. 4, "Compression").  init: payload of nbits bits (bits past the end
 * read as zero). */
int lmgc_decode_init(lmgc_decoder* st, const uint8_t* payload, uint64_t nbits);
/* Decode one symbol with model row cdf_row[nsym+1]; *sym_out gets the bin. */
int lmgc_decode_symbol(lmgc_decoder* st, const uint32_t* cdf_row, int32_t nsym,
                       int32_t* sym_out);

/* -------------------------------------------------------------- container */
/*
 * Container: what the compression rate of Eq. 3 counts (all its bytes).
 * Windows are coded independently (Sec. 4: the stream is split into
 * windows of the LM's context), so the header records each window's bit
 * count.  Layout (little-endian): 128-byte header
 *   0 "LMGC" | 4 u16 version=1 | 6 u16 header bytes=128 | 8 u64 model tag |
 *   16 u64 n_values | 24 u8 bytes_per_value | 25 u8 bytes_per_group |
 *   26 u8 msb_first | 27 u8 nsym (A + 1) | 28 u32 W | 32 u32 total |
 *   36 u32 n_windows | 40 i32 bos | 44 i32 pad | 48 i32 sep | 52 i32 hex[16] |
 *   116 u32 sep2_id + 1 (0: none) | 120 u32 renorm | 124..127 zero
 * then u32 bits[n_windows], then the payloads, each ceil(bits/8) bytes.
 */
#define LMGC_HEADER_BYTES 128

/* Upper bound of the container size for n_values values. */
size_t lmgc_container_bound(int64_t n_values, const lmgc_serial_params* p);

/* Device workspace bytes lmgc_compress / lmgc_decode need (the larger of
 * the two: compression holds one batch's activations, decoding the K/V
 * cache of up to min(batch, 32) windows). */
size_t lmgc_codec_workspace(const lmgc_model* m, int64_t n_values, const lmgc_serial_params* p,
                            int32_t batch);

/*
 * LM-GC compression (Sec. 4, Fig. 1: serialise, LM tables, arithmetic
 * coding, per window).  Compress d_values (device) into a container at out (host).  Windows
 * [first_window, first_window + n_windows) are coded (n_windows < 0: all
 * windows from first_window on); the header records all of the vector's
 * windows only when the whole vector is coded.  batch windows per LM call;
 * host coding of one batch overlaps the GPU work of the next.  Synchronises
 * stream before returning.  Errors: EINVAL, ESIZE (cap or ws), EDEVICE.
 */
int lmgc_compress(const lmgc_model* m, const void* d_values, int64_t n_values,
                  const lmgc_serial_params* p, uint32_t total, int32_t batch,
                  uint64_t model_tag, int64_t first_window, int64_t n_windows,
                  void* d_ws, size_t ws_bytes, uint8_t* out, size_t cap, size_t* used,
                  void* stream);

/*
 * LM-GC decompression (Sec. 4, "Compression": the LM is replayed from BOS
 * and each decoded token is fed back).  Decompress a whole-vector container
 * into values_out (host, n_values * bytes_per_value bytes).  Decodes groups of min(batch, 32) windows token by
 * token from BOS: each step computes the next position's tables of the
 * group through the K/V cache (as lmgc_probs_stepwise, bit for bit the
 * encoder's tables), the host decodes one symbol per window and its token
 * is the next step's input.  expect_tag
 * must equal the header's model tag.  Errors: ECORRUPT (bad container,
 * escape symbol, malformed stream, tag mismatch), ESIZE, EDEVICE.
 */
int lmgc_decode(const lmgc_model* m, const uint8_t* container, size_t bytes, int32_t batch,
                uint64_t expect_tag, void* d_ws, size_t ws_bytes, void* values_out,
                void* stream);

/* Parse a container header (the layout above): n_values and windows, for
 * sizing buffers.  Errors: ECORRUPT. */
int lmgc_container_info(const uint8_t* container, size_t bytes, int64_t* n_values,
                        int32_t* bytes_per_value, int64_t* n_windows, uint64_t* model_tag);

/* ----------------------------------------------------- kernel-level calls */
/*
 * C[M, N] (float32) = A[M, K] * B[N, K]^T with bfloat16 A, B (bit patterns)
 * and float32 accumulation: the matrix-product kernel of the decoder's
 * projections (Sec. 5.1 LLMs), exposed for parity tests at full size.
 * K must be a multiple of 64 and N of 256; A is [M, K] row-major, B is
 * [N, K] row-major, C is [M, N] row-major.  GPU, async.
 */
int lmgc_op_gemm_bf16(const uint16_t* d_a, const uint16_t* d_b, float* d_c, int32_t M,
                      int32_t N, int32_t K, void* stream);

/*
 * The decoder's own matrix-product instantiations (weights in MFMA blocks,
 * fused epilogues), exposed so that tests check what the model runs at full
 * size.  B [N, K] bfloat16 in MFMA blocks (lmgc_op_block_weights), A [M, K]
 * row-major bfloat16, float32 accumulation, K % 64 == 0, N % 256 == 0.
 *   LMGC_OP_STORE:  out float32 [M, N] = A B^T (the operand ring holds B
 *                   when N >= 2K, as for the LM head and QKV projections);
 *   LMGC_OP_RESID:  out float32 [M, N] += A B^T (the residual add of the O
 *                   and down projections; the ring holds A);
 *   LMGC_OP_SWIGLU: out bfloat16 [M, N/2]: B's rows are gate and up rows
 *                   interleaved in groups of 32 (row 64g + t is gate feature
 *                   32g + t, row 64g + 32 + t its up row, t < 32), and
 *                   out[m, f] = bf16(silu(gate) * up) (the gate/up
 *                   projection, the dominant kernel).
 * Pointers 16-byte aligned, device memory.  GPU, async.  Errors: EINVAL.
 */
enum { LMGC_OP_STORE = 0, LMGC_OP_RESID = 1, LMGC_OP_SWIGLU = 2 };
int lmgc_op_gemm_bf16_blocked(const uint16_t* d_a, const uint16_t* d_b, void* d_out, int32_t M,
                              int32_t N, int32_t K, int32_t kind, void* stream);
/* Row-major bfloat16 [N, K] -> MFMA blocks (16 rows x 32 k per 1 KB, lane
 * order of the 16x16x32 MFMA's B operand): the layout the model keeps its
 * weights in.  N % 16 == 0, K % 32 == 0, d_dst != d_src.  GPU, async. */
int lmgc_op_block_weights(const uint16_t* d_src, uint16_t* d_dst, int32_t N, int32_t K,
                          void* stream);

/*
 * Causal attention kernel of the decoder on bfloat16 operands (the model
 * the paper runs, Sec. 5.1): q [B, Hq, W, hd] and k [B, Hkv, W, hd]
 * row-major, v given TRANSPOSED as vt [B, Hkv, hd, W] (the layout the bf16
 * decoder keeps V in) -> o [B*W, Hq*hd] bfloat16, softmax of q.k/sqrt(hd)
 * over keys <= query; query head h reads kv head h*Hkv/Hq.  hd in {64, 128},
 * W % 8 == 0 (else LMGC_EUNSUPPORTED).  All pointers are device memory the
 * caller owns, 16-byte aligned.  GPU, async on `stream`.
 */
int lmgc_op_attention_bf16(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_vt,
                           uint16_t* d_o, int32_t B, int32_t Hq, int32_t Hkv, int32_t W,
                           int32_t hd, void* stream);

/* ------------------------------------------------------------------ timing */
/*
 * Per-kernel timing with HIP events recorded around each launch lmgc_probs
 * makes on its stream.  Kinds index the dominant kernels.
 */
enum {
  LMGC_K_EMBED = 0,
  LMGC_K_NORM = 1,
  LMGC_K_GEMM_QKV = 2,
  LMGC_K_ATTN = 3,
  LMGC_K_GEMM_O = 4,
  LMGC_K_GEMM_UP = 5,   /* gate/up with SwiGLU (LLAMA) or fc with GELU (GPT2) */
  LMGC_K_GEMM_DOWN = 6,
  LMGC_K_GEMM_HEAD = 7,
  LMGC_K_LSE_CDF = 8,
  LMGC_K_COUNT = 9
};
/* Enable (1) or disable (0) timing and clear the accumulated times. */
int lmgc_timing_enable(int32_t enable);
/*
 * Record events only around launches of the kinds in `kind_mask` (bit k =
 * kind k; the default is every kind).  Each recorded pair adds a little
 * time between launches, so a timed run can restrict them to the kernel it
 * reports.  EINVAL if the mask has no valid kind.
 */
int lmgc_timing_kinds(uint32_t kind_mask);
/* Synchronise pending events; total milliseconds and launches of `kind`. */
int lmgc_timing_read(int32_t kind, double* total_ms, int64_t* count);
/* Algorithmic floating-point operations of one lmgc_probs call, by kind. */
double lmgc_probs_flops(const lmgc_model* m, int32_t B, int32_t W, int32_t kind);

#ifdef __cplusplus
}
#endif
#endif /* LMGC_H */
