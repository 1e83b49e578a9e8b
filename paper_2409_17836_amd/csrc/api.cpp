// C ABI of liblmgc: argument checking, model repacking, the per-window LM
// forward that produces the coder's tables (lmgc_probs), and the codec
// drivers (lmgc_compress / lmgc_decode) that chain serialisation, the LM and
// the host arithmetic coder.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <exception>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "common.h"
#include "host.h"

namespace lmgc {

// ------------------------------------------------------------------ errors
static thread_local char g_err[512] = "";

int set_error(int code, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return code;
}
void clear_error() { g_err[0] = 0; }

#define HIP_OK(expr)                                                                  \
  do {                                                                                \
    hipError_t e_ = (expr);                                                           \
    if (e_ != hipSuccess)                                                             \
      return set_error(LMGC_EDEVICE, "%s: %s (%s)", __func__, hipGetErrorString(e_), #expr); \
  } while (0)

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
static int64_t round_up(int64_t x, int64_t a) { return (x + a - 1) / a * a; }

// ------------------------------------------------------------ serial params
// Token ids of the coder's alphabet bins (hex digits, then the separator
// tokens); returns the alphabet size (17 or 18).
static int alphabet(const lmgc_serial_params& p, int32_t* ids) {
  for (int i = 0; i < 16; i++) ids[i] = p.hex_ids[i];
  ids[16] = p.sep_id;
  if (p.sep2_id >= 0) {
    ids[17] = p.sep2_id;
    return 18;
  }
  return 17;
}

static int check_serial(const lmgc_serial_params* p, int vocab) {
  if (!p) return set_error(LMGC_EINVAL, "serial params are NULL");
  if (p->bytes_per_value != 1 && p->bytes_per_value != 2 && p->bytes_per_value != 4)
    return set_error(LMGC_EINVAL, "bytes_per_value must be 1, 2 or 4");
  if (p->bytes_per_group < 0 || p->bytes_per_group > 255)
    return set_error(LMGC_EINVAL, "bytes_per_group must be in [0, 255]");
  if (p->msb_first != 0 && p->msb_first != 1) return set_error(LMGC_EINVAL, "msb_first must be 0 or 1");
  if (p->window <= 0) return set_error(LMGC_EINVAL, "window must be positive");
  if (p->sep2_id < -1) return set_error(LMGC_EINVAL, "sep2_id must be -1 (none) or a token id");
  if (p->renorm != 0 && p->renorm != 1) return set_error(LMGC_EINVAL, "renorm must be 0 or 1");
  int32_t ids[LMGC_NALPHA_MAX];
  const int na = alphabet(*p, ids);
  for (int a = 0; a < na; a++)
    for (int b2 = a + 1; b2 < na; b2++)
      if (ids[a] == ids[b2]) return set_error(LMGC_EINVAL, "alphabet token ids must be distinct (id %d twice)", ids[a]);
  if (vocab > 0) {
    const int32_t ext[2] = {p->bos_id, p->pad_id};
    for (int i = 0; i < 2; i++)
      if (ext[i] < 0 || ext[i] >= vocab) return set_error(LMGC_EINVAL, "token id %d outside the vocabulary", ext[i]);
    for (int a = 0; a < na; a++)
      if (ids[a] < 0 || ids[a] >= vocab) return set_error(LMGC_EINVAL, "alphabet id %d outside the vocabulary", ids[a]);
  }
  return LMGC_OK;
}

// ------------------------------------------------------------------ timing
struct Timing {
  std::mutex mu;
  bool on = false;
  uint32_t mask = (1u << LMGC_K_COUNT) - 1;  // kinds whose launches get events
  std::vector<std::pair<hipEvent_t, hipEvent_t>> pending[LMGC_K_COUNT];
  double ms[LMGC_K_COUNT] = {};
  int64_t count[LMGC_K_COUNT] = {};
  std::vector<hipEvent_t> pool;
};
static Timing g_timing;

struct ScopedTimer {
  int kind;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  ScopedTimer(int k, hipStream_t st) : kind(k), s(st) {
    std::lock_guard<std::mutex> g(g_timing.mu);
    if (!g_timing.on || !((g_timing.mask >> kind) & 1u)) return;
    for (hipEvent_t* e : {&a, &b}) {
      if (!g_timing.pool.empty()) {
        *e = g_timing.pool.back();
        g_timing.pool.pop_back();
      } else if (hipEventCreate(e) != hipSuccess) {
        *e = nullptr;
      }
    }
    if (a) hipEventRecord(a, s);
  }
  ~ScopedTimer() {
    if (!a || !b) return;
    hipEventRecord(b, s);
    std::lock_guard<std::mutex> g(g_timing.mu);
    g_timing.pending[kind].push_back({a, b});
  }
};

// ------------------------------------------------------------------- model
struct Layer {
  const void *n1 = nullptr, *n1b = nullptr, *n2 = nullptr, *n2b = nullptr;
  const void *wqkv = nullptr, *bqkv = nullptr, *wo = nullptr, *bo = nullptr;
  const void *wup = nullptr, *bup = nullptr, *wdown = nullptr, *bdown = nullptr;
};

}  // namespace lmgc

struct lmgc_model {
  lmgc_model_config cfg;
  int hd = 0, act = 0, tile = 0;  // head dim, activation bytes, N padding
  int n_qkv = 0, n_qkv_pad = 0, n_up = 0, n_up_pad = 0, d_pad = 0, v_pad = 0;
  const void *tok_emb = nullptr, *pos_emb = nullptr, *final_g = nullptr, *final_b = nullptr;
  const void* head = nullptr;        // [v_pad, d]
  const float2* rope = nullptr;      // [max_pos, hd/2]
  std::vector<lmgc::Layer> layers;
  std::vector<void*> allocs;
  ~lmgc_model() {
    for (void* p : allocs) hipFree(p);
  }
};

namespace lmgc {

static int check_config(const lmgc_model_config* c) {
  if (!c) return set_error(LMGC_EINVAL, "config is NULL");
  if (c->arch != LMGC_ARCH_LLAMA && c->arch != LMGC_ARCH_GPT2) return set_error(LMGC_EINVAL, "unknown arch");
  if (c->dtype != LMGC_DTYPE_F32 && c->dtype != LMGC_DTYPE_BF16) return set_error(LMGC_EINVAL, "unknown dtype");
  if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->d_ff <= 0 ||
      c->vocab <= 0 || c->max_pos <= 0)
    return set_error(LMGC_EINVAL, "sizes must be positive");
  if (c->d_model % c->n_heads) return set_error(LMGC_EINVAL, "d_model must be a multiple of n_heads");
  if (c->n_heads % c->n_kv_heads) return set_error(LMGC_EINVAL, "n_heads must be a multiple of n_kv_heads");
  if (c->arch == LMGC_ARCH_GPT2 && c->n_kv_heads != c->n_heads)
    return set_error(LMGC_EINVAL, "GPT2 arch has n_kv_heads == n_heads");
  const int hd = c->d_model / c->n_heads;
  if (c->d_model % 64 || c->d_ff % 64) return set_error(LMGC_EINVAL, "d_model and d_ff must be multiples of 64");
  if (c->dtype == LMGC_DTYPE_BF16 && hd != 64 && hd != 128)
    return set_error(LMGC_EUNSUPPORTED, "bf16 models need head_dim 64 or 128 (got %d)", hd);
  if (c->dtype == LMGC_DTYPE_F32 && (hd % 16 || hd > 64))
    return set_error(LMGC_EUNSUPPORTED, "f32 models need head_dim in {16, 32, 48, 64} (got %d)", hd);
  if (c->arch == LMGC_ARCH_LLAMA && ((c->n_kv_heads * hd) % 64))
    return set_error(LMGC_EUNSUPPORTED, "n_kv_heads * head_dim must be a multiple of 64");
  if (c->d_model > 8192) return set_error(LMGC_EUNSUPPORTED, "d_model above 8192");
  return LMGC_OK;
}

struct TensorInfo {
  std::string name;
  int ndim;
  int64_t shape[2];
};

static std::vector<TensorInfo> manifest(const lmgc_model_config& c) {
  std::vector<TensorInfo> m;
  const int64_t d = c.d_model, hd = c.d_model / c.n_heads, F = c.d_ff, V = c.vocab;
  auto add = [&](std::string n, int64_t a, int64_t b = -1) {
    TensorInfo t;
    t.name = n;
    t.ndim = b < 0 ? 1 : 2;
    t.shape[0] = a;
    t.shape[1] = b < 0 ? 1 : b;
    m.push_back(t);
  };
  if (c.arch == LMGC_ARCH_LLAMA) {
    add("tok_emb", V, d);
    for (int l = 0; l < c.n_layers; l++) {
      const std::string p = "l" + std::to_string(l) + ".";
      add(p + "attn_norm", d);
      add(p + "wq", c.n_heads * hd, d);
      add(p + "wk", c.n_kv_heads * hd, d);
      add(p + "wv", c.n_kv_heads * hd, d);
      add(p + "wo", d, c.n_heads * hd);
      add(p + "ffn_norm", d);
      add(p + "w_gate", F, d);
      add(p + "w_up", F, d);
      add(p + "w_down", d, F);
    }
    add("final_norm", d);
    add("lm_head", V, d);
  } else {
    add("wte", V, d);
    add("wpe", c.max_pos, d);
    for (int l = 0; l < c.n_layers; l++) {
      const std::string p = "l" + std::to_string(l) + ".";
      add(p + "ln1_g", d);
      add(p + "ln1_b", d);
      add(p + "w_qkv", 3 * d, d);
      add(p + "b_qkv", 3 * d);
      add(p + "w_o", d, d);
      add(p + "b_o", d);
      add(p + "ln2_g", d);
      add(p + "ln2_b", d);
      add(p + "w_fc", F, d);
      add(p + "b_fc", F);
      add(p + "w_proj", d, F);
      add(p + "b_proj", d);
    }
    add("lnf_g", d);
    add("lnf_b", d);
  }
  return m;
}

// Device copy of a whole tensor.
static int copy_tensor(lmgc_model* m, const void* src, size_t bytes, hipStream_t s, const void** out) {
  void* p = nullptr;
  HIP_OK(hipMalloc(&p, std::max<size_t>(bytes, 256)));
  m->allocs.push_back(p);
  HIP_OK(hipMemcpyAsync(p, src, bytes, hipMemcpyDeviceToDevice, s));
  *out = p;
  return LMGC_OK;
}

// Repack rows: out[r] = srcs[idx[r] >> 28][idx[r] & 0x0fffffff] (or zeros);
// bf16 matrices are written in MFMA blocks.
static int gather_tensor(lmgc_model* m, GatherSrcs srcs, const std::vector<int32_t>& idx, int cols,
                         hipStream_t s, std::vector<void*>& temps, const void** out) {
  const size_t row_bytes = (size_t)cols * m->act;
  void* p = nullptr;
  HIP_OK(hipMalloc(&p, idx.size() * row_bytes));
  m->allocs.push_back(p);
  void* d_idx = nullptr;
  HIP_OK(hipMalloc(&d_idx, idx.size() * sizeof(int32_t)));
  temps.push_back(d_idx);
  HIP_OK(hipMemcpyAsync(d_idx, idx.data(), idx.size() * sizeof(int32_t), hipMemcpyHostToDevice, s));
  // bf16 weights go to MFMA blocks (the layout the matrix kernels take B in)
  if (m->act == 2)
    HIP_OK(launch_gather_rows_blocked(srcs, (const int32_t*)d_idx, (int)idx.size(), cols, p, s));
  else
    HIP_OK(launch_gather_rows(srcs, (const int32_t*)d_idx, (int)idx.size(), cols, m->act, p, s));
  *out = p;
  return LMGC_OK;
}

static std::vector<int32_t> natural_rows(int n, int n_pad, int src = 0) {
  std::vector<int32_t> idx(n_pad, -1);
  for (int r = 0; r < n; r++) idx[r] = (src << 28) | r;
  return idx;
}

// Column c of a q or k segment -> (head, dim) row of the original weight:
// 64-column group g holds rotation pairs g*32 .. g*32+31, column g*64 + t is
// dim i of pair P = g*32 + t, column g*64 + 32 + t its partner i + hd/2.
static int rope_row(int c, int hd) {
  const int g = c / 64, w = c % 64, half = w / 32, P = g * 32 + w % 32;
  const int head = P / (hd / 2), i = P % (hd / 2);
  return head * hd + i + half * (hd / 2);
}

static int create_model(const lmgc_model_config* cfg, const void* const* w, hipStream_t s,
                        lmgc_model** out) {
  int rc = check_config(cfg);
  if (rc) return rc;
  if (!w || !out) return set_error(LMGC_EINVAL, "NULL weights or output handle");
  const auto man = manifest(*cfg);
  for (size_t i = 0; i < man.size(); i++)
    if (!w[i]) return set_error(LMGC_EINVAL, "weight %zu (%s) is NULL", i, man[i].name.c_str());

  lmgc_model* m = new lmgc_model();
  m->cfg = *cfg;
  const lmgc_model_config& c = *cfg;
  m->hd = c.d_model / c.n_heads;
  m->act = c.dtype == LMGC_DTYPE_BF16 ? 2 : 4;
  m->tile = c.dtype == LMGC_DTYPE_BF16 ? 256 : 64;
  const int d = c.d_model, hd = m->hd, F = c.d_ff;
  m->n_qkv = (c.n_heads + 2 * c.n_kv_heads) * hd;
  m->n_qkv_pad = (int)round_up(m->n_qkv, m->tile);
  m->n_up = c.arch == LMGC_ARCH_LLAMA ? 2 * F : F;
  m->n_up_pad = (int)round_up(m->n_up, m->tile);
  m->d_pad = (int)round_up(d, m->tile);
  m->v_pad = (int)round_up(c.vocab, m->tile);
  std::vector<void*> temps;
  // Frees the repack temporaries on every exit, and the model too unless it
  // was handed out (also when a host allocation throws).
  struct Cleanup {
    std::vector<void*>& temps;
    lmgc_model*& m;
    ~Cleanup() {
      for (void* p : temps) hipFree(p);
      delete m;
    }
  } cleanup{temps, m};
  auto fail = [](int code) { return code; };
  auto vec_bytes = [&](int64_t n) { return (size_t)n * m->act; };
  size_t k = 0;  // manifest cursor
  if (c.arch == LMGC_ARCH_LLAMA) {
    if ((rc = copy_tensor(m, w[k++], vec_bytes((int64_t)c.vocab * d), s, &m->tok_emb))) return fail(rc);
    m->layers.resize(c.n_layers);
    for (int l = 0; l < c.n_layers; l++) {
      Layer& L = m->layers[l];
      const void *n1 = w[k], *wq = w[k + 1], *wk = w[k + 2], *wv = w[k + 3], *wo = w[k + 4], *n2 = w[k + 5],
                 *wg = w[k + 6], *wu = w[k + 7], *wd = w[k + 8];
      k += 9;
      if ((rc = copy_tensor(m, n1, vec_bytes(d), s, &L.n1))) return fail(rc);
      if ((rc = copy_tensor(m, n2, vec_bytes(d), s, &L.n2))) return fail(rc);
      std::vector<int32_t> idx(m->n_qkv_pad, -1);
      const int sq = c.n_heads * hd, sk = c.n_kv_heads * hd;
      for (int r = 0; r < sq; r++) idx[r] = (0 << 28) | rope_row(r, hd);
      for (int r = 0; r < sk; r++) idx[sq + r] = (1 << 28) | rope_row(r, hd);
      for (int r = 0; r < sk; r++) idx[sq + sk + r] = (2 << 28) | r;
      if ((rc = gather_tensor(m, GatherSrcs{{wq, wk, wv, nullptr}}, idx, d, s, temps, &L.wqkv))) return fail(rc);
      if ((rc = gather_tensor(m, GatherSrcs{{wo, nullptr, nullptr, nullptr}}, natural_rows(d, m->d_pad), sq, s,
                              temps, &L.wo)))
        return fail(rc);
      std::vector<int32_t> gu(m->n_up_pad, -1);
      for (int r = 0; r < 2 * F; r++) {
        const int g = r / 64, t = r % 64;
        gu[r] = t < 32 ? ((0 << 28) | (g * 32 + t)) : ((1 << 28) | (g * 32 + t - 32));
      }
      if ((rc = gather_tensor(m, GatherSrcs{{wg, wu, nullptr, nullptr}}, gu, d, s, temps, &L.wup))) return fail(rc);
      if ((rc = gather_tensor(m, GatherSrcs{{wd, nullptr, nullptr, nullptr}}, natural_rows(d, m->d_pad), F, s,
                              temps, &L.wdown)))
        return fail(rc);
    }
    if ((rc = copy_tensor(m, w[k++], vec_bytes(d), s, &m->final_g))) return fail(rc);
    if ((rc = gather_tensor(m, GatherSrcs{{w[k++], nullptr, nullptr, nullptr}}, natural_rows(c.vocab, m->v_pad),
                            d, s, temps, &m->head)))
      return fail(rc);
    // RoPE table in double, rounded to float
    std::vector<float2> tab((size_t)c.max_pos * (hd / 2));
    for (int p = 0; p < c.max_pos; p++)
      for (int i = 0; i < hd / 2; i++) {
        const double ang = (double)p * pow((double)c.rope_theta, -2.0 * i / hd);
        tab[(size_t)p * (hd / 2) + i] = make_float2((float)cos(ang), (float)sin(ang));
      }
    void* pr = nullptr;
    if (hipMalloc(&pr, tab.size() * sizeof(float2)) != hipSuccess) return fail(set_error(LMGC_ENOMEM, "rope table"));
    m->allocs.push_back(pr);
    if (hipMemcpyAsync(pr, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice, s) != hipSuccess ||
        hipStreamSynchronize(s) != hipSuccess)
      return fail(set_error(LMGC_EDEVICE, "rope table upload"));
    m->rope = (const float2*)pr;
  } else {
    const void* wte = w[k++];
    if ((rc = copy_tensor(m, wte, vec_bytes((int64_t)c.vocab * d), s, &m->tok_emb))) return fail(rc);
    if ((rc = copy_tensor(m, w[k++], vec_bytes((int64_t)c.max_pos * d), s, &m->pos_emb))) return fail(rc);
    m->layers.resize(c.n_layers);
    for (int l = 0; l < c.n_layers; l++) {
      Layer& L = m->layers[l];
      if ((rc = copy_tensor(m, w[k + 0], vec_bytes(d), s, &L.n1))) return fail(rc);
      if ((rc = copy_tensor(m, w[k + 1], vec_bytes(d), s, &L.n1b))) return fail(rc);
      if ((rc = gather_tensor(m, GatherSrcs{{w[k + 2], nullptr, nullptr, nullptr}},
                              natural_rows(3 * d, m->n_qkv_pad), d, s, temps, &L.wqkv)))
        return fail(rc);
      if ((rc = copy_tensor(m, w[k + 3], vec_bytes(3 * d), s, &L.bqkv))) return fail(rc);
      if ((rc = gather_tensor(m, GatherSrcs{{w[k + 4], nullptr, nullptr, nullptr}}, natural_rows(d, m->d_pad), d,
                              s, temps, &L.wo)))
        return fail(rc);
      if ((rc = copy_tensor(m, w[k + 5], vec_bytes(d), s, &L.bo))) return fail(rc);
      if ((rc = copy_tensor(m, w[k + 6], vec_bytes(d), s, &L.n2))) return fail(rc);
      if ((rc = copy_tensor(m, w[k + 7], vec_bytes(d), s, &L.n2b))) return fail(rc);
      if ((rc = gather_tensor(m, GatherSrcs{{w[k + 8], nullptr, nullptr, nullptr}}, natural_rows(F, m->n_up_pad),
                              d, s, temps, &L.wup)))
        return fail(rc);
      if ((rc = copy_tensor(m, w[k + 9], vec_bytes(F), s, &L.bup))) return fail(rc);
      if ((rc = gather_tensor(m, GatherSrcs{{w[k + 10], nullptr, nullptr, nullptr}}, natural_rows(d, m->d_pad), F,
                              s, temps, &L.wdown)))
        return fail(rc);
      if ((rc = copy_tensor(m, w[k + 11], vec_bytes(d), s, &L.bdown))) return fail(rc);
      k += 12;
    }
    if ((rc = copy_tensor(m, w[k++], vec_bytes(d), s, &m->final_g))) return fail(rc);
    if ((rc = copy_tensor(m, w[k++], vec_bytes(d), s, &m->final_b))) return fail(rc);
    if ((rc = gather_tensor(m, GatherSrcs{{wte, nullptr, nullptr, nullptr}}, natural_rows(c.vocab, m->v_pad), d,
                            s, temps, &m->head)))
      return fail(rc);
  }
  if (hipStreamSynchronize(s) != hipSuccess) return fail(set_error(LMGC_EDEVICE, "model repack failed"));
  *out = m;
  m = nullptr;  // owned by the caller now
  return LMGC_OK;
}

// ------------------------------------------------------- probs workspace
struct ProbsWs {
  float* h;
  void *a, *q, *k, *v, *o, *ff;
  float* za;         // [M, LMGC_NALPHA_MAX] alphabet logits
  float2* part;      // [M, v_pad / 64] log-sum-exp partials of the LM head
  void* head_alpha;  // [tile, d] alphabet rows of the LM head (renormalised tables)
  size_t bytes;
};

static ProbsWs carve(const lmgc_model* m, int B, int W, char* base) {
  const lmgc_model_config& c = m->cfg;
  const size_t M = (size_t)B * W, A = 256;
  ProbsWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, A);
    return p;
  };
  w.h = (float*)take(M * c.d_model * 4);
  w.a = take(M * std::max(c.d_model, c.n_heads * m->hd) * m->act);
  w.q = take(M * c.n_heads * m->hd * m->act);
  w.k = take(M * c.n_kv_heads * m->hd * m->act);
  w.v = take(M * c.n_kv_heads * m->hd * m->act);
  w.o = take(M * c.n_heads * m->hd * m->act);
  w.ff = take(M * c.d_ff * m->act);
  w.za = (float*)take(M * LMGC_NALPHA_MAX * 4);
  w.part = (float2*)take(M * (m->v_pad / 64) * sizeof(float2));
  w.head_alpha = take((size_t)m->tile * c.d_model * m->act);
  w.bytes = off;
  return w;
}

// ---------------------------------------------------------------- forward
// Activation buffers of one forward pass.  kc[l] / vc[l]: layer l's K and V
// (V^T for bf16 models) in [B, Hkv, W, hd] ([B, Hkv, hd, W]) layout; a batch
// of whole windows may point every layer at one buffer, a decoding step
// keeps one per layer (the cache).
struct FwdBufs {
  float* h;
  void *a, *q, *o, *ff;
  float* za;
  float2* part;
  void* head_alpha;
  void* const* kc;
  void* const* vc;
};

// The decoder over B windows of W tokens.  dpos < 0: all W positions of each
// window (rows b*W + j; tok is [B, W]).  dpos >= 0: one decoding step, the
// row of position dpos of each window (rows b; tok[b] is the token at
// dpos - 1; layers read K and V of earlier positions from the cache and add
// their own).  Every kernel computes a row exactly as in the full pass, so
// the step's tables equal the full pass's row dpos bit for bit.
static int forward(const lmgc_model* m, const int32_t* tok, int B, int W, int dpos, const lmgc_serial_params* p,
                   uint32_t total, const FwdBufs& f, uint32_t* cdf, float* logp, hipStream_t s) {
  const lmgc_model_config& c = m->cfg;
  const bool step = dpos >= 0;
  const int M = step ? B : B * W, d = c.d_model, hd = m->hd, F = c.d_ff;
  const bool bf = c.dtype == LMGC_DTYPE_BF16;
  const bool llama = c.arch == LMGC_ARCH_LLAMA;
  auto gemm = [&](const void* A, const void* Bw, int Npad, int K, EpiArgs e) {
    e.step = step ? 1 : 0;
    e.dpos = step ? dpos : 0;
    if (!bf) return launch_gemm_f32((const float*)A, (const float*)Bw, M, Npad, K, e, s);
    return step ? launch_gemm_bf16_rows((const uint16_t*)A, (const uint16_t*)Bw, M, Npad, K, e, s)
                : launch_gemm_bf16((const uint16_t*)A, (const uint16_t*)Bw, M, Npad, K, e, s);
  };
  {
    ScopedTimer t(LMGC_K_EMBED, s);
    HIP_OK(launch_embed(tok, B, W, p->bos_id, m->tok_emb, m->pos_emb, d, c.vocab, c.dtype, dpos, f.h, s));
  }
  for (int l = 0; l < c.n_layers; l++) {
    const Layer& L = m->layers[l];
    {
      ScopedTimer t(LMGC_K_NORM, s);
      HIP_OK(launch_norm(f.h, M, d, L.n1, L.n1b, !llama, c.norm_eps, c.dtype, f.a, s));
    }
    {
      ScopedTimer t(LMGC_K_GEMM_QKV, s);
      EpiArgs e = {};
      e.kind = llama ? EPI_QKV_ROPE : EPI_QKV_BIAS;
      e.M = M;
      e.N = m->n_qkv;
      e.bias = L.bqkv;
      e.q = f.q;
      e.k = f.kc[l];
      e.v = f.vc[l];
      e.W = W;
      e.Hq = c.n_heads;
      e.Hkv = c.n_kv_heads;
      e.hd = hd;
      e.rope = m->rope;
      HIP_OK(gemm(f.a, L.wqkv, m->n_qkv_pad, d, e));
    }
    {
      ScopedTimer t(LMGC_K_ATTN, s);
      if (bf)
        HIP_OK(launch_attention_bf16((const uint16_t*)f.q, (const uint16_t*)f.kc[l], (const uint16_t*)f.vc[l],
                                     (uint16_t*)f.o, B, c.n_heads, c.n_kv_heads, W, hd, dpos, s));
      else
        HIP_OK(launch_attention_f32((const float*)f.q, (const float*)f.kc[l], (const float*)f.vc[l], (float*)f.o,
                                    B, c.n_heads, c.n_kv_heads, W, hd, dpos, s));
    }
    {
      ScopedTimer t(LMGC_K_GEMM_O, s);
      EpiArgs e = {};
      e.kind = EPI_RESID;
      e.M = M;
      e.N = d;
      e.c = f.h;
      e.ldc = d;
      e.bias = L.bo;
      HIP_OK(gemm(f.o, L.wo, m->d_pad, c.n_heads * hd, e));
    }
    {
      ScopedTimer t(LMGC_K_NORM, s);
      HIP_OK(launch_norm(f.h, M, d, L.n2, L.n2b, !llama, c.norm_eps, c.dtype, f.a, s));
    }
    {
      ScopedTimer t(LMGC_K_GEMM_UP, s);
      EpiArgs e = {};
      e.kind = llama ? EPI_SWIGLU : EPI_BIAS_GELU;
      e.M = M;
      e.N = m->n_up;
      e.bias = L.bup;
      e.out = f.ff;
      e.ld_out = F;
      HIP_OK(gemm(f.a, L.wup, m->n_up_pad, d, e));
    }
    {
      ScopedTimer t(LMGC_K_GEMM_DOWN, s);
      EpiArgs e = {};
      e.kind = EPI_RESID;
      e.M = M;
      e.N = d;
      e.c = f.h;
      e.ldc = d;
      e.bias = L.bdown;
      HIP_OK(gemm(f.ff, L.wdown, m->d_pad, F, e));
    }
  }
  {
    ScopedTimer t(LMGC_K_NORM, s);
    HIP_OK(launch_norm(f.h, M, d, m->final_g, m->final_b, !llama, c.norm_eps, c.dtype, f.a, s));
  }
  // LM head (Sec. 4, "Compression": the coder's distribution is the LM's
  // softmax over the whole vocabulary).  The logits stay in registers: the
  // head GEMM's epilogue writes each row's log-sum-exp partial per 64-column
  // group and the alphabet logits, and launch_head_tables merges the
  // partials in a fixed order into the LSE and quantises the table.
  int32_t ids[LMGC_NALPHA_MAX];
  const int na = alphabet(*p, ids);
  EpiArgs e = {};
  e.kind = EPI_HEAD;
  e.M = M;
  e.za = f.za;
  e.ld_za = LMGC_NALPHA_MAX;
  e.n_alpha = na;
  if (p->renorm) {
    // Renormalised tables need only the alphabet's logits: the LM head is
    // cut to its A alphabet rows (one N tile, columns 0..A-1), and the LSE
    // runs over them.
    ScopedTimer t(LMGC_K_GEMM_HEAD, s);
    HIP_OK(launch_alpha_head(m->head, ids, na, m->tile, d, m->act, f.head_alpha, s));
    for (int a = 0; a < na; a++) e.alpha_ids[a] = a;
    e.N = na;
    e.part = nullptr;
    e.ngroups = m->tile / 64;
    HIP_OK(gemm(f.a, f.head_alpha, m->tile, d, e));
  } else {
    ScopedTimer t(LMGC_K_GEMM_HEAD, s);
    for (int a = 0; a < na; a++) e.alpha_ids[a] = ids[a];
    e.N = c.vocab;
    e.part = f.part;
    e.ngroups = m->v_pad / 64;
    HIP_OK(gemm(f.a, m->head, m->v_pad, d, e));
  }
  {
    ScopedTimer t(LMGC_K_LSE_CDF, s);
    HIP_OK(launch_head_tables(f.part, m->v_pad / 64, f.za, LMGC_NALPHA_MAX, M, na, total, p->renorm, cdf,
                              logp, s));
  }
  return LMGC_OK;
}

static int run_probs(const lmgc_model* m, const int32_t* tok, int B, int W, const lmgc_serial_params* p,
                     uint32_t total, uint32_t* cdf, float* logp, void* ws, size_t ws_bytes, hipStream_t s) {
  if (!m) return set_error(LMGC_EINVAL, "model is NULL");
  const lmgc_model_config& c = m->cfg;
  int rc = check_serial(p, c.vocab);
  if (rc) return rc;
  if (B <= 0 || W <= 0) return set_error(LMGC_EINVAL, "B and W must be positive");
  if (W > c.max_pos) return set_error(LMGC_EINVAL, "W=%d exceeds the model's max_pos=%d", W, c.max_pos);
  if (c.dtype == LMGC_DTYPE_BF16 && W % 8) return set_error(LMGC_EUNSUPPORTED, "bf16 models need W %% 8 == 0");
  if ((int64_t)B * W > (1 << 26)) return set_error(LMGC_EUNSUPPORTED, "B*W above 2^26 rows");
  if (total < 2 * LMGC_NSYM_MAX || total > (1u << 24)) return set_error(LMGC_EINVAL, "total must be in [38, 2^24]");
  if (!tok || !cdf || !ws) return set_error(LMGC_EINVAL, "NULL device buffer");
  ProbsWs w = carve(m, B, W, (char*)ws);
  if (ws_bytes < w.bytes) return set_error(LMGC_ESIZE, "workspace too small: %zu < %zu", ws_bytes, w.bytes);

  std::vector<void*> kc(c.n_layers, w.k), vc(c.n_layers, w.v);
  const FwdBufs f = {w.h, w.a, w.q, w.o, w.ff, w.za, w.part, w.head_alpha, kc.data(), vc.data()};
  return forward(m, tok, B, W, -1, p, total, f, cdf, logp, s);
}

static double probs_flops(const lmgc_model* m, int B, int W, int kind) {
  if (!m) return 0.0;
  const lmgc_model_config& c = m->cfg;
  const double M = (double)B * W, d = c.d_model, hd = m->hd, F = c.d_ff, L = c.n_layers;
  switch (kind) {
    case LMGC_K_GEMM_QKV: return L * 2 * M * d * m->n_qkv;
    case LMGC_K_GEMM_O: return L * 2 * M * (c.n_heads * hd) * d;
    case LMGC_K_GEMM_UP: return L * 2 * M * d * m->n_up;
    case LMGC_K_GEMM_DOWN: return L * 2 * M * F * d;
    case LMGC_K_GEMM_HEAD: return 2 * M * d * c.vocab;
    case LMGC_K_ATTN: return L * (double)B * c.n_heads * 2.0 * hd * (double)W * (W + 1);
    default: return 0.0;
  }
}

// ------------------------------------------------------------ codec driver
// --------------------------------------------------- decoding-step workspace
// One decoding step works on compact rows (one per window) and keeps every
// layer's K and V of the window group in a cache; q keeps the [B, Hq, W, hd]
// layout the attention kernel reads (only the current position is written).
constexpr int kStepMaxB = 32;  // rows of the one-row GEMM kernel

struct StepWs {
  float* h;
  void *a, *q, *o, *ff;
  float* za;         // [B, LMGC_NALPHA_MAX] alphabet logits
  float2* part;      // [B, v_pad / 64] log-sum-exp partials of the LM head
  void* head_alpha;  // [tile, d] alphabet rows of the LM head (renormalised tables)
  int32_t* tok;     // [B] input token of the step (the previous position's)
  uint32_t* cdf;    // [B, A + 2] (A: alphabet size)
  float* logp;      // [B, A]
  char* zero_from;  // q and the caches: cleared for every window group
  size_t zero_bytes, bytes;
  std::vector<void*> kc, vc;
};

static StepWs carve_step(const lmgc_model* m, int B, int W, char* base) {
  const lmgc_model_config& c = m->cfg;
  StepWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  const size_t act = m->act, hq = (size_t)c.n_heads * m->hd, hkv = (size_t)c.n_kv_heads * m->hd;
  w.h = (float*)take((size_t)B * c.d_model * 4);
  w.a = take((size_t)B * std::max<size_t>(c.d_model, hq) * act);
  w.o = take((size_t)B * hq * act);
  w.ff = take((size_t)B * c.d_ff * act);
  w.za = (float*)take((size_t)B * LMGC_NALPHA_MAX * 4);
  w.part = (float2*)take((size_t)B * (m->v_pad / 64) * sizeof(float2));
  w.head_alpha = take((size_t)m->tile * c.d_model * act);
  w.tok = (int32_t*)take((size_t)B * 4);
  w.cdf = (uint32_t*)take((size_t)B * (LMGC_NSYM_MAX + 1) * 4);
  w.logp = (float*)take((size_t)B * LMGC_NALPHA_MAX * 4);
  const size_t z0 = off;
  w.q = take((size_t)B * W * hq * act);
  for (int l = 0; l < c.n_layers; l++) {
    w.kc.push_back(take((size_t)B * W * hkv * act));
    w.vc.push_back(take((size_t)B * W * hkv * act));
  }
  w.zero_from = base ? base + z0 : nullptr;
  w.zero_bytes = off - z0;
  w.bytes = off;
  return w;
}

static int check_step(const lmgc_model* m, int B, int W, const lmgc_serial_params* p, uint32_t total) {
  if (!m) return set_error(LMGC_EINVAL, "model is NULL");
  int rc = check_serial(p, m->cfg.vocab);
  if (rc) return rc;
  if (B <= 0 || B > kStepMaxB || W <= 0) return set_error(LMGC_EINVAL, "need 0 < B <= %d and W > 0", kStepMaxB);
  if (W > m->cfg.max_pos) return set_error(LMGC_EINVAL, "W=%d exceeds the model's max_pos=%d", W, m->cfg.max_pos);
  if (m->cfg.dtype == LMGC_DTYPE_BF16 && W % 8) return set_error(LMGC_EUNSUPPORTED, "bf16 models need W %% 8 == 0");
  if (total < 2 * LMGC_NSYM_MAX || total > (1u << 24)) return set_error(LMGC_EINVAL, "total must be in [38, 2^24]");
  return LMGC_OK;
}

// One decoding step at position j of every window of the group (w.tok holds
// the tokens at j - 1); tables land in w.cdf (and w.logp).
static int run_step(const lmgc_model* m, StepWs& w, int B, int W, int j, const lmgc_serial_params* p,
                    uint32_t total, bool want_logp, hipStream_t s) {
  const FwdBufs f = {w.h, w.a, w.q, w.o, w.ff, w.za, w.part, w.head_alpha, w.kc.data(), w.vc.data()};
  return forward(m, w.tok, B, W, j, p, total, f, w.cdf, want_logp ? w.logp : nullptr, s);
}

// lmgc_probs computed one position at a time through the cache, with the
// given tokens as the decoded prefix.
static int run_stepwise(const lmgc_model* m, const int32_t* tok, int B, int W, const lmgc_serial_params* p,
                        uint32_t total, uint32_t* cdf, float* logp, void* ws, size_t ws_bytes, hipStream_t s) {
  int rc = check_step(m, B, W, p, total);
  if (rc) return rc;
  if (!tok || !cdf || !ws) return set_error(LMGC_EINVAL, "NULL device buffer");
  StepWs w = carve_step(m, B, W, (char*)ws);
  if (ws_bytes < w.bytes) return set_error(LMGC_ESIZE, "workspace too small: %zu < %zu", ws_bytes, w.bytes);
  int32_t ids[LMGC_NALPHA_MAX];
  const size_t na = alphabet(*p, ids), tw = na + 2;  // alphabet, table width
  HIP_OK(hipMemsetAsync(w.zero_from, 0, w.zero_bytes, s));
  for (int j = 0; j < W; j++) {
    if (j > 0) HIP_OK(hipMemcpy2DAsync(w.tok, 4, tok + (j - 1), (size_t)W * 4, 4, B, hipMemcpyDeviceToDevice, s));
    if ((rc = run_step(m, w, B, W, j, p, total, logp != nullptr, s))) return rc;
    HIP_OK(hipMemcpy2DAsync(cdf + (size_t)j * tw, (size_t)W * tw * 4, w.cdf, tw * 4, tw * 4, B,
                            hipMemcpyDeviceToDevice, s));
    if (logp)
      HIP_OK(hipMemcpy2DAsync(logp + (size_t)j * na, (size_t)W * na * 4, w.logp, na * 4, na * 4, B,
                              hipMemcpyDeviceToDevice, s));
  }
  return LMGC_OK;
}

struct CodecWs {
  int32_t* tok;
  uint8_t* sym;
  uint32_t* cdf;
  char* probs;
  size_t probs_bytes, bytes;
};

static CodecWs carve_codec(const lmgc_model* m, int B, int W, char* base) {
  CodecWs c;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  const size_t M = (size_t)B * W;
  c.tok = (int32_t*)take(M * 4);
  c.sym = (uint8_t*)take(M);
  c.cdf = (uint32_t*)take(M * (LMGC_NSYM_MAX + 1) * 4);
  c.probs_bytes = carve(m, B, W, nullptr).bytes;
  c.probs = take(c.probs_bytes);
  c.bytes = off;
  return c;
}

struct PinnedBuf {
  void* p = nullptr;
  ~PinnedBuf() {
    if (p) hipHostFree(p);
  }
};

static int compress(const lmgc_model* m, const void* d_values, int64_t n_values, const lmgc_serial_params* p,
                    uint32_t total, int32_t B, uint64_t tag, int64_t first_window, int64_t n_windows, void* ws,
                    size_t ws_bytes, uint8_t* out, size_t cap, size_t* used, hipStream_t s) {
  if (!m) return set_error(LMGC_EINVAL, "model is NULL");
  int rc = check_serial(p, m->cfg.vocab);
  if (rc) return rc;
  if (!d_values && n_values > 0) return set_error(LMGC_EINVAL, "values are NULL");
  if (!out || !used || n_values < 0 || n_values > LMGC_MAX_VALUES || B <= 0)
    return set_error(LMGC_EINVAL, "bad arguments");
  const int W = p->window;
  const int64_t nt = num_tokens(n_values, *p);
  const int64_t nw_all = (nt + W - 1) / W;
  if (n_windows < 0) n_windows = nw_all - first_window;
  if (first_window < 0 || n_windows < 0 || first_window + n_windows > nw_all)
    return set_error(LMGC_EINVAL, "window range [%lld, +%lld) outside [0, %lld)", (long long)first_window,
                     (long long)n_windows, (long long)nw_all);
  CodecWs cw = carve_codec(m, B, W, (char*)ws);
  if (ws_bytes < cw.bytes) return set_error(LMGC_ESIZE, "codec workspace too small: %zu < %zu", ws_bytes, cw.bytes);
  const size_t head_bytes = LMGC_HEADER_BYTES + 4 * (size_t)n_windows;
  if (cap < head_bytes) return set_error(LMGC_ESIZE, "output buffer too small for the header");

  const size_t M = (size_t)B * W;
  int32_t alpha_ids[LMGC_NALPHA_MAX];
  const int nsym = alphabet(*p, alpha_ids) + 1;  // coder bins incl. escape
  PinnedBuf hc[2], hs[2];
  for (int i = 0; i < 2; i++) {
    HIP_OK(hipHostMalloc(&hc[i].p, M * (nsym + 1) * 4, hipHostMallocDefault));
    HIP_OK(hipHostMalloc(&hs[i].p, M, hipHostMallocDefault));
  }
  hipEvent_t ev[2];
  HIP_OK(hipEventCreateWithFlags(&ev[0], hipEventDisableTiming));
  if (hipEventCreateWithFlags(&ev[1], hipEventDisableTiming) != hipSuccess) {
    hipEventDestroy(ev[0]);
    return set_error(LMGC_EDEVICE, "event create");
  }
  struct EvGuard {
    hipEvent_t* e;
    ~EvGuard() {
      hipEventDestroy(e[0]);
      hipEventDestroy(e[1]);
    }
  } evg{ev};

  std::vector<uint32_t> bits(n_windows, 0);
  std::vector<int32_t> lens(B);
  size_t pos = head_bytes;
  const int64_t nbatch = (n_windows + B - 1) / B;
  auto encode_batch = [&](int64_t b) -> int {
    const int64_t w0 = b * B;
    const int nb = (int)std::min<int64_t>(B, n_windows - w0);
    for (int i = 0; i < nb; i++) {
      const int64_t gw = first_window + w0 + i;
      lens[i] = (int)std::min<int64_t>(W, nt - gw * W);
    }
    size_t u = 0;
    int r = encode_windows((const uint32_t*)hc[b & 1].p, nsym, (const uint8_t*)hs[b & 1].p, lens.data(), nb, W,
                           out + pos, cap - pos, bits.data() + w0, &u, 0);
    if (r) return r;
    pos += u;
    return LMGC_OK;
  };
  for (int64_t b = 0; b < nbatch; b++) {
    const int64_t w0 = b * B;
    const int nb = (int)std::min<int64_t>(B, n_windows - w0);
    HIP_OK(launch_serialize(d_values, n_values, *p, first_window + w0, nb, cw.tok, cw.sym, s));
    rc = run_probs(m, cw.tok, nb, W, p, total, cw.cdf, nullptr, cw.probs, cw.probs_bytes, s);
    if (rc) return rc;
    HIP_OK(hipMemcpyAsync(hc[b & 1].p, cw.cdf, (size_t)nb * W * (nsym + 1) * 4, hipMemcpyDeviceToHost, s));
    HIP_OK(hipMemcpyAsync(hs[b & 1].p, cw.sym, (size_t)nb * W, hipMemcpyDeviceToHost, s));
    HIP_OK(hipEventRecord(ev[b & 1], s));
    if (b > 0) {
      HIP_OK(hipEventSynchronize(ev[(b - 1) & 1]));
      if ((rc = encode_batch(b - 1))) return rc;
    }
  }
  if (nbatch > 0) {
    HIP_OK(hipEventSynchronize(ev[(nbatch - 1) & 1]));
    if ((rc = encode_batch(nbatch - 1))) return rc;
  }
  HIP_OK(hipStreamSynchronize(s));
  ContainerHeader h;
  h.model_tag = tag;
  h.n_values = n_values;
  h.p = *p;
  h.total = total;
  h.n_windows = n_windows;
  write_header(out, h);
  if (n_windows) memcpy(out + LMGC_HEADER_BYTES, bits.data(), 4 * (size_t)n_windows);
  *used = pos;
  return LMGC_OK;
}

static int decode(const lmgc_model* m, const uint8_t* buf, size_t bytes, int32_t B, uint64_t tag, void* ws,
                  size_t ws_bytes, void* values_out, hipStream_t s) {
  if (!m || !buf || !values_out || B <= 0) return set_error(LMGC_EINVAL, "bad arguments");
  ContainerHeader h;
  int rc = read_header(buf, bytes, &h);
  if (rc) return rc;
  if (h.model_tag != tag) return set_error(LMGC_ECORRUPT, "container model tag does not match");
  if ((rc = check_serial(&h.p, m->cfg.vocab))) return rc;
  const int W = h.p.window;
  const int64_t nt = num_tokens(h.n_values, h.p);
  const int G = std::min(B, kStepMaxB);  // windows decoded together
  if ((rc = check_step(m, G, W, &h.p, h.total))) return rc;
  StepWs sw = carve_step(m, G, W, (char*)ws);
  if (ws_bytes < sw.bytes) return set_error(LMGC_ESIZE, "codec workspace too small: %zu < %zu", ws_bytes, sw.bytes);
  std::vector<uint32_t> bits(h.n_windows);
  if (h.n_windows) memcpy(bits.data(), buf + LMGC_HEADER_BYTES, 4 * (size_t)h.n_windows);
  std::vector<size_t> off(h.n_windows + 1);
  off[0] = LMGC_HEADER_BYTES + 4 * (size_t)h.n_windows;
  for (int64_t w = 0; w < h.n_windows; w++) off[w + 1] = off[w] + (bits[w] + 7) / 8;
  if (off[h.n_windows] > bytes) return set_error(LMGC_ECORRUPT, "container: truncated payload");

  std::vector<uint8_t> sym((size_t)std::max<int64_t>(nt, 1));
  std::vector<int32_t> id_of(LMGC_NALPHA_MAX);
  const int na = alphabet(h.p, id_of.data()), nsym = na + 1;
  std::vector<uint32_t> rows((size_t)G * (nsym + 1));
  std::vector<int32_t> col(G);
  std::vector<lmgc_decoder> dec(G);
  // Window groups, token by token from BOS: one decoding step gives every
  // window of the group the table of its next position, the host decodes
  // the symbols, and their tokens are the next step's input.
  for (int64_t w0 = 0; w0 < h.n_windows; w0 += G) {
    const int nb = (int)std::min<int64_t>(G, h.n_windows - w0);
    std::vector<int> len(nb);
    int maxlen = 0;
    for (int i = 0; i < nb; i++) {
      len[i] = (int)std::min<int64_t>(W, nt - (w0 + i) * W);
      maxlen = std::max(maxlen, len[i]);
      decoder_init(&dec[i], buf + off[w0 + i], bits[w0 + i]);
    }
    HIP_OK(hipMemsetAsync(sw.zero_from, 0, sw.zero_bytes, s));
    for (int j = 0; j < maxlen; j++) {
      if ((rc = run_step(m, sw, nb, W, j, &h.p, h.total, false, s))) return rc;
      HIP_OK(hipMemcpyAsync(rows.data(), sw.cdf, (size_t)nb * (nsym + 1) * 4, hipMemcpyDeviceToHost, s));
      HIP_OK(hipStreamSynchronize(s));
      for (int i = 0; i < nb; i++) {
        col[i] = h.p.pad_id;
        if (j >= len[i]) continue;
        int32_t b = 0;
        if ((rc = decoder_symbol(&dec[i], rows.data() + (size_t)i * (nsym + 1), nsym, &b))) return rc;
        if (b >= na) return set_error(LMGC_ECORRUPT, "escape symbol decoded (window %lld, position %d)",
                                              (long long)(w0 + i), j);
        sym[(size_t)(w0 + i) * W + j] = (uint8_t)b;
        col[i] = id_of[b];
      }
      HIP_OK(hipMemcpyAsync(sw.tok, col.data(), (size_t)nb * 4, hipMemcpyHostToDevice, s));
    }
  }
  HIP_OK(hipStreamSynchronize(s));
  return deserialize_bins(sym.data(), nt, h.n_values, h.p, (uint8_t*)values_out);
}

// Host allocations (std containers, threads) can throw; the ABI reports
// LMGC_ENOMEM (or LMGC_EDEVICE for any other host exception) instead of
// letting an exception cross it.
template <class F>
static auto guarded(F&& f) -> decltype(f()) {
  try {
    return f();
  } catch (const std::bad_alloc&) {
    return (decltype(f()))set_error(LMGC_ENOMEM, "host memory allocation failed");
  } catch (const std::exception& e) {
    return (decltype(f()))set_error(LMGC_EDEVICE, "host error: %s", e.what());
  }
}

}  // namespace lmgc

// ===================================================================== ABI
using namespace lmgc;

extern "C" {

const char* lmgc_last_error(void) { return g_err; }
const char* lmgc_version(void) { return "lmgc 0.1 gfx950"; }

int32_t lmgc_alphabet_size(const lmgc_serial_params* p) {
  clear_error();
  if (check_serial(p, 0)) return -1;
  int32_t ids[LMGC_NALPHA_MAX];
  return alphabet(*p, ids);
}

int64_t lmgc_num_tokens(int64_t n_values, const lmgc_serial_params* p) {
  if (check_serial(p, 0) || n_values < 0) return -1;
  return num_tokens(n_values, *p);
}

int64_t lmgc_num_windows(int64_t n_values, const lmgc_serial_params* p) {
  const int64_t nt = lmgc_num_tokens(n_values, p);
  if (nt < 0) return -1;
  return (nt + p->window - 1) / p->window;
}

int lmgc_serialize(const void* d_values, int64_t n_values, const lmgc_serial_params* p, int64_t first_window,
                   int64_t n_windows, int32_t* d_tokens, uint8_t* d_sym, void* stream) {
  clear_error();
  int rc = check_serial(p, 0);
  if (rc) return rc;
  if (n_values < 0 || (n_values > 0 && !d_values) || !d_tokens) return set_error(LMGC_EINVAL, "bad buffers");
  if (((uintptr_t)d_tokens & 15) || ((uintptr_t)d_sym & 3))
    return set_error(LMGC_EINVAL, "d_tokens must be 16-byte and d_sym 4-byte aligned");
  const int64_t nw = lmgc_num_windows(n_values, p);
  if (nw < 0) return set_error(LMGC_EINVAL, "n_values above LMGC_MAX_VALUES");
  if (first_window < 0 || n_windows < 0 || first_window + n_windows > nw)
    return set_error(LMGC_EINVAL, "window range outside the stream");
  hipError_t e = launch_serialize(d_values, n_values, *p, first_window, n_windows, d_tokens, d_sym,
                                  (hipStream_t)stream);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "serialize launch: %s", hipGetErrorString(e));
  return LMGC_OK;
}

int lmgc_deserialize(const uint8_t* sym, int64_t n_tokens, int64_t n_values, const lmgc_serial_params* p,
                     void* values_out) {
  clear_error();
  int rc = check_serial(p, 0);
  if (rc) return rc;
  if (n_values < 0 || n_tokens < 0 || (n_tokens && !sym) || (n_values && !values_out))
    return set_error(LMGC_EINVAL, "bad buffers");
  return deserialize_bins(sym, n_tokens, n_values, *p, (uint8_t*)values_out);
}

static int check_lossy_vec(const float* d_values, int64_t n_values, const void* d_out) {
  if (n_values < 0 || n_values > INT32_MAX) return set_error(LMGC_EINVAL, "n_values must be in [0, 2^31 - 1]");
  if (n_values > 0 && (!d_values || !d_out)) return set_error(LMGC_EINVAL, "bad buffers");
  if (((uintptr_t)d_values & 15) || ((uintptr_t)d_out & 15))
    return set_error(LMGC_EINVAL, "device buffers must be 16-byte aligned");
  return LMGC_OK;
}

static int check_lossy_ws(const void* ws, size_t bytes) {
  if (!ws || bytes < lossy_workspace_bytes())
    return set_error(LMGC_ESIZE, "lossy workspace needs %zu bytes", lossy_workspace_bytes());
  if ((uintptr_t)ws & 15) return set_error(LMGC_EINVAL, "workspace must be 16-byte aligned");
  return LMGC_OK;
}

int64_t lmgc_keep_count(int64_t n_values, int32_t percent) {
  clear_error();
  if (n_values < 0 || n_values > INT32_MAX) return set_error(LMGC_EINVAL, "n_values must be in [0, 2^31 - 1]");
  if (percent < 0 || percent > 100) return set_error(LMGC_EINVAL, "percent must be in [0, 100]");
  return n_values * percent / 100;  // < 2^38: no overflow
}

int64_t lmgc_lossy_workspace(int64_t n_values) {
  clear_error();
  if (n_values < 0 || n_values > INT32_MAX) return set_error(LMGC_EINVAL, "n_values must be in [0, 2^31 - 1]");
  return (int64_t)lossy_workspace_bytes();
}

static int check_topk(const float* d_values, int64_t n_values, int64_t k, const float* d_out) {
  int rc = check_lossy_vec(d_values, n_values, d_out);
  if (rc) return rc;
  if (k < 0) return set_error(LMGC_EINVAL, "k must be >= 0");
  if (d_out != d_values && n_values > 0 &&
      (const char*)d_out < (const char*)(d_values + n_values) && (const char*)d_values < (const char*)(d_out + n_values))
    return set_error(LMGC_EINVAL, "d_out overlaps d_values without being equal to it");
  return LMGC_OK;
}

int lmgc_sparsify_topk(const float* d_values, int64_t n_values, int64_t k, float* d_out, void* d_workspace,
                       size_t workspace_bytes, void* stream) {
  clear_error();
  int rc = check_topk(d_values, n_values, k, d_out);
  if (rc) return rc;
  if (n_values == 0) return LMGC_OK;
  if (k > 0 && (rc = check_lossy_ws(d_workspace, workspace_bytes))) return rc;
  hipError_t e = launch_sparsify_topk(d_values, n_values, k, d_out, d_workspace, (hipStream_t)stream);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "sparsify launch: %s", hipGetErrorString(e));
  return LMGC_OK;
}

int lmgc_sparsify_topk_noalloc(const float* d_values, int64_t n_values, int64_t k, float* d_out, void* stream) {
  clear_error();
  int rc = check_topk(d_values, n_values, k, d_out);
  if (rc) return rc;
  if (n_values == 0) return LMGC_OK;
  void* ws = nullptr;
  size_t cap = 0;
  hipError_t e = lossy_scratch(&ws, &cap);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "library scratch: %s", hipGetErrorString(e));
  if (lossy_workspace_bytes() > cap)
    return set_error(LMGC_ESIZE, "top-k needs %zu bytes of scratch, the library holds %zu", lossy_workspace_bytes(),
                     cap);
  e = launch_sparsify_topk(d_values, n_values, k, d_out, ws, (hipStream_t)stream);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "sparsify launch: %s", hipGetErrorString(e));
  return LMGC_OK;
}

int lmgc_quantize_linear(const float* d_values, int64_t n_values, int32_t bits, void* d_indices, float* min_max,
                         void* d_workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  int rc = check_lossy_vec(d_values, n_values, d_indices);
  if (rc) return rc;
  if (bits < 1 || bits > 16) return set_error(LMGC_EINVAL, "bits must be in [1, 16]");
  if (n_values == 0) {
    if (min_max) min_max[0] = min_max[1] = 0.0f;
    return LMGC_OK;
  }
  if ((rc = check_lossy_ws(d_workspace, workspace_bytes))) return rc;
  hipStream_t s = (hipStream_t)stream;
  LossyMinMax* slot = lossy_minmax_slot(d_workspace);
  hipError_t e = launch_minmax(d_values, n_values, d_workspace, slot, s);
  LossyMinMax mm{};
  if (e == hipSuccess) e = hipMemcpyAsync(&mm, slot, sizeof(mm), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "quantize min/max: %s", hipGetErrorString(e));
  if (mm.nonfinite) return set_error(LMGC_EINVAL, "values hold %u NaN or infinite entries", mm.nonfinite);
  e = launch_quantize_linear(d_values, n_values, bits, mm.mn, mm.mx, d_indices, s);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "quantize launch: %s", hipGetErrorString(e));
  if (min_max) {
    min_max[0] = mm.mn;
    min_max[1] = mm.mx;
  }
  return LMGC_OK;
}

int lmgc_sign_pack(const float* d_values, int64_t n_values, uint8_t* d_out, void* stream) {
  clear_error();
  if (n_values < 0 || n_values > INT32_MAX) return set_error(LMGC_EINVAL, "n_values must be in [0, 2^31 - 1]");
  if (n_values > 0 && (!d_values || !d_out)) return set_error(LMGC_EINVAL, "bad buffers");
  if ((uintptr_t)d_values & 15) return set_error(LMGC_EINVAL, "d_values must be 16-byte aligned");
  hipError_t e = launch_sign_pack(d_values, n_values, d_out, (hipStream_t)stream);
  if (e != hipSuccess) return set_error(LMGC_EDEVICE, "sign pack launch: %s", hipGetErrorString(e));
  return LMGC_OK;
}

int32_t lmgc_model_num_tensors(const lmgc_model_config* cfg) {
  clear_error();
  if (check_config(cfg)) return -1;
  return guarded([&] { return (int32_t)manifest(*cfg).size(); });
}

int lmgc_model_tensor_info(const lmgc_model_config* cfg, int32_t index, char* name, size_t name_cap,
                           int32_t* ndim, int64_t shape[2]) {
  clear_error();
  int rc = check_config(cfg);
  if (rc) return rc;
  std::vector<TensorInfo> man;
  if ((rc = guarded([&] { man = manifest(*cfg); return LMGC_OK; }))) return rc;
  if (index < 0 || (size_t)index >= man.size()) return set_error(LMGC_EINVAL, "tensor index out of range");
  const TensorInfo& t = man[index];
  if (name && name_cap) {
    strncpy(name, t.name.c_str(), name_cap - 1);
    name[name_cap - 1] = 0;
  }
  if (ndim) *ndim = t.ndim;
  if (shape) {
    shape[0] = t.shape[0];
    shape[1] = t.shape[1];
  }
  return LMGC_OK;
}

int lmgc_model_create(const lmgc_model_config* cfg, const void* const* d_weights, void* stream, lmgc_model** out) {
  clear_error();
  return guarded([&] { return create_model(cfg, d_weights, (hipStream_t)stream, out); });
}

void lmgc_model_destroy(lmgc_model* m) { delete m; }

size_t lmgc_probs_workspace(const lmgc_model* m, int32_t B, int32_t W) {
  if (!m || B <= 0 || W <= 0) return 0;
  return carve(m, B, W, nullptr).bytes;
}

int lmgc_probs(const lmgc_model* m, const int32_t* d_tokens, int32_t B, int32_t W, const lmgc_serial_params* p,
               uint32_t total, uint32_t* d_cdf, float* d_logp, void* d_ws, size_t ws_bytes, void* stream) {
  clear_error();
  return guarded([&] { return run_probs(m, d_tokens, B, W, p, total, d_cdf, d_logp, d_ws, ws_bytes, (hipStream_t)stream); });
}

size_t lmgc_encode_bound(int32_t n_win, int32_t W) {
  if (n_win <= 0 || W <= 0) return 0;
  return (size_t)n_win * encode_bound_bytes(W);
}

int lmgc_encode(const uint32_t* cdf, int32_t nsym, const uint8_t* sym, const int32_t* len, int32_t n_win,
                int32_t W, uint8_t* out, size_t cap, uint32_t* bits, size_t* used, int32_t n_threads) {
  clear_error();
  if (nsym < 2 || nsym > 256 || n_win < 0 || W <= 0 || !used || (n_win > 0 && (!cdf || !sym || !len || !bits)))
    return set_error(LMGC_EINVAL, "lmgc_encode: bad arguments");
  if (n_win > 0 && !out) return set_error(LMGC_EINVAL, "lmgc_encode: NULL output");
  return guarded([&] { return encode_windows(cdf, nsym, sym, len, n_win, W, out, cap, bits, used, n_threads); });
}

int lmgc_decode_init(lmgc_decoder* st, const uint8_t* payload, uint64_t nbits) {
  clear_error();
  if (!st || (nbits && !payload)) return set_error(LMGC_EINVAL, "lmgc_decode_init: bad arguments");
  return decoder_init(st, payload, nbits);
}

int lmgc_decode_symbol(lmgc_decoder* st, const uint32_t* cdf_row, int32_t nsym, int32_t* sym_out) {
  if (!st || !cdf_row || !sym_out || nsym < 2 || nsym > 256)
    return set_error(LMGC_EINVAL, "lmgc_decode_symbol: bad arguments");
  return decoder_symbol(st, cdf_row, nsym, sym_out);
}

size_t lmgc_container_bound(int64_t n_values, const lmgc_serial_params* p) {
  const int64_t nw = lmgc_num_windows(n_values, p);
  if (nw < 0) return 0;
  return LMGC_HEADER_BYTES + (size_t)nw * (4 + encode_bound_bytes(p->window));
}

size_t lmgc_codec_workspace(const lmgc_model* m, int64_t n_values, const lmgc_serial_params* p, int32_t batch) {
  (void)n_values;
  if (!m || !p || batch <= 0 || p->window <= 0) return 0;
  return std::max(carve_codec(m, batch, p->window, nullptr).bytes,
                  carve_step(m, std::min(batch, kStepMaxB), p->window, nullptr).bytes);
}

size_t lmgc_step_workspace(const lmgc_model* m, int32_t B, int32_t W) {
  if (!m || B <= 0 || B > kStepMaxB || W <= 0) return 0;
  return carve_step(m, B, W, nullptr).bytes;
}

int lmgc_probs_stepwise(const lmgc_model* m, const int32_t* d_tokens, int32_t B, int32_t W,
                        const lmgc_serial_params* p, uint32_t total, uint32_t* d_cdf, float* d_logp, void* d_ws,
                        size_t ws_bytes, void* stream) {
  clear_error();
  return guarded([&] { return run_stepwise(m, d_tokens, B, W, p, total, d_cdf, d_logp, d_ws, ws_bytes, (hipStream_t)stream); });
}

int lmgc_compress(const lmgc_model* m, const void* d_values, int64_t n_values, const lmgc_serial_params* p,
                  uint32_t total, int32_t batch, uint64_t model_tag, int64_t first_window, int64_t n_windows,
                  void* d_ws, size_t ws_bytes, uint8_t* out, size_t cap, size_t* used, void* stream) {
  clear_error();
  return guarded([&] {
    return compress(m, d_values, n_values, p, total, batch, model_tag, first_window, n_windows, d_ws, ws_bytes, out,
                    cap, used, (hipStream_t)stream);
  });
}

int lmgc_decode(const lmgc_model* m, const uint8_t* container, size_t bytes, int32_t batch, uint64_t expect_tag,
                void* d_ws, size_t ws_bytes, void* values_out, void* stream) {
  clear_error();
  return guarded([&] { return decode(m, container, bytes, batch, expect_tag, d_ws, ws_bytes, values_out, (hipStream_t)stream); });
}

int lmgc_container_info(const uint8_t* container, size_t bytes, int64_t* n_values, int32_t* bytes_per_value,
                        int64_t* n_windows, uint64_t* model_tag) {
  clear_error();
  ContainerHeader h;
  int rc = read_header(container, bytes, &h);
  if (rc) return rc;
  if (n_values) *n_values = h.n_values;
  if (bytes_per_value) *bytes_per_value = h.p.bytes_per_value;
  if (n_windows) *n_windows = h.n_windows;
  if (model_tag) *model_tag = h.model_tag;
  return LMGC_OK;
}

int lmgc_op_gemm_bf16(const uint16_t* d_a, const uint16_t* d_b, float* d_c, int32_t M, int32_t N, int32_t K,
                      void* stream) {
  clear_error();
  if (!d_a || !d_b || !d_c || M < 0 || N <= 0 || K <= 0) return set_error(LMGC_EINVAL, "bad arguments");
  if (K % 64 || N % 256) return set_error(LMGC_EINVAL, "need K %% 64 == 0 and N %% 256 == 0");
  EpiArgs e = {};
  e.kind = EPI_STORE_F32;
  e.M = M;
  e.N = N;
  e.c = d_c;
  e.ldc = N;
  hipError_t err = launch_gemm_bf16(d_a, d_b, M, N, K, e, (hipStream_t)stream, false);
  if (err != hipSuccess) return set_error(LMGC_EDEVICE, "gemm launch: %s", hipGetErrorString(err));
  return LMGC_OK;
}

int lmgc_op_block_weights(const uint16_t* d_src, uint16_t* d_dst, int32_t N, int32_t K, void* stream) {
  clear_error();
  if (!d_src || !d_dst || N <= 0 || K <= 0) return set_error(LMGC_EINVAL, "bad arguments");
  if (N % 16 || K % 32) return set_error(LMGC_EINVAL, "need N %% 16 == 0 and K %% 32 == 0");
  if (((uintptr_t)d_src & 15) || ((uintptr_t)d_dst & 15)) return set_error(LMGC_EINVAL, "pointers must be 16-byte aligned");
  if (d_src == d_dst) return set_error(LMGC_EINVAL, "d_dst must not be d_src");
  hipError_t err = launch_gather_rows_blocked(GatherSrcs{{d_src, nullptr, nullptr, nullptr}}, nullptr, N, K, d_dst,
                                              (hipStream_t)stream);
  if (err != hipSuccess) return set_error(LMGC_EDEVICE, "block launch: %s", hipGetErrorString(err));
  return LMGC_OK;
}

int lmgc_op_gemm_bf16_blocked(const uint16_t* d_a, const uint16_t* d_b, void* d_out, int32_t M, int32_t N,
                              int32_t K, int32_t kind, void* stream) {
  clear_error();
  if (!d_a || !d_b || !d_out || M < 0 || N <= 0 || K <= 0) return set_error(LMGC_EINVAL, "bad arguments");
  if (K % 64 || N % 256) return set_error(LMGC_EINVAL, "need K %% 64 == 0 and N %% 256 == 0");
  if (((uintptr_t)d_a & 15) || ((uintptr_t)d_b & 15) || ((uintptr_t)d_out & 15))
    return set_error(LMGC_EINVAL, "pointers must be 16-byte aligned");
  EpiArgs e = {};
  e.M = M;
  e.N = N;
  switch (kind) {
    case LMGC_OP_STORE:
      e.kind = EPI_STORE_F32;
      e.c = (float*)d_out;
      e.ldc = N;
      break;
    case LMGC_OP_RESID:
      e.kind = EPI_RESID;
      e.c = (float*)d_out;
      e.ldc = N;
      break;
    case LMGC_OP_SWIGLU:
      e.kind = EPI_SWIGLU;
      e.out = d_out;
      e.ld_out = N / 2;
      break;
    default:
      return set_error(LMGC_EINVAL, "unknown kind %d", kind);
  }
  hipError_t err = launch_gemm_bf16(d_a, d_b, M, N, K, e, (hipStream_t)stream, true);
  if (err != hipSuccess) return set_error(LMGC_EDEVICE, "gemm launch: %s", hipGetErrorString(err));
  return LMGC_OK;
}

int lmgc_op_attention_bf16(const uint16_t* d_q, const uint16_t* d_k, const uint16_t* d_vt, uint16_t* d_o,
                           int32_t B, int32_t Hq, int32_t Hkv, int32_t W, int32_t hd, void* stream) {
  clear_error();
  if (!d_q || !d_k || !d_vt || !d_o || B <= 0 || W <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv)
    return set_error(LMGC_EINVAL, "bad arguments");
  if ((hd != 64 && hd != 128) || W % 8) return set_error(LMGC_EUNSUPPORTED, "need hd in {64, 128} and W %% 8 == 0");
  hipError_t err = launch_attention_bf16(d_q, d_k, d_vt, d_o, B, Hq, Hkv, W, hd, -1, (hipStream_t)stream);
  if (err != hipSuccess) return set_error(LMGC_EDEVICE, "attention launch: %s", hipGetErrorString(err));
  return LMGC_OK;
}

int lmgc_timing_enable(int32_t enable) {
  return guarded([&] {
  std::lock_guard<std::mutex> g(g_timing.mu);
  g_timing.on = enable != 0;
  for (int k = 0; k < LMGC_K_COUNT; k++) {
    for (auto& pr : g_timing.pending[k]) {
      hipEventSynchronize(pr.second);
      g_timing.pool.push_back(pr.first);
      g_timing.pool.push_back(pr.second);
    }
    g_timing.pending[k].clear();
    g_timing.ms[k] = 0;
    g_timing.count[k] = 0;
  }
  return LMGC_OK;
  });
}

int lmgc_timing_kinds(uint32_t kind_mask) {
  kind_mask &= (1u << LMGC_K_COUNT) - 1;
  if (!kind_mask) return set_error(LMGC_EINVAL, "lmgc_timing_kinds: no valid kind in the mask");
  std::lock_guard<std::mutex> g(g_timing.mu);
  g_timing.mask = kind_mask;
  return LMGC_OK;
}

int lmgc_timing_read(int32_t kind, double* total_ms, int64_t* count) {
  if (kind < 0 || kind >= LMGC_K_COUNT) return set_error(LMGC_EINVAL, "bad kernel kind");
  return guarded([&] {
  std::lock_guard<std::mutex> g(g_timing.mu);
  for (int k = 0; k < LMGC_K_COUNT; k++) {
    for (auto& pr : g_timing.pending[k]) {
      float ms = 0.f;
      if (hipEventSynchronize(pr.second) == hipSuccess && hipEventElapsedTime(&ms, pr.first, pr.second) == hipSuccess) {
        g_timing.ms[k] += ms;
        g_timing.count[k] += 1;
      }
      g_timing.pool.push_back(pr.first);
      g_timing.pool.push_back(pr.second);
    }
    g_timing.pending[k].clear();
  }
  if (total_ms) *total_ms = g_timing.ms[kind];
  if (count) *count = g_timing.count[kind];
  return LMGC_OK;
  });
}

double lmgc_probs_flops(const lmgc_model* m, int32_t B, int32_t W, int32_t kind) {
  return probs_flops(m, B, W, kind);
}

}  // extern "C"
