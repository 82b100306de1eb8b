// C ABI of the patch-parallel DiT denoising step: context, weight loading,
// argument validation and the per-step launch sequence (Algorithm 1: one-step
// inference on the device's band with the stale buffer, then the buffer
// update; the scheduler update of §I with Lemma 1's coefficient).
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/orch.h"
#include "common.h"
#include "kernels.h"

using namespace orch;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(ORCH_EHIP, "%s: %s", what, hipGetErrorString(e));
}

#define HIP_TRY(expr, what)                  \
  do {                                       \
    hipError_t _e = (expr);                  \
    if (_e != hipSuccess) return hip_fail(_e, what); \
  } while (0)

size_t esize(int dtype) { return dtype == ORCH_BF16 ? 2 : 4; }

bool ranges_overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

float bf16_bits_to_float(uint16_t v) {
  uint32_t u = (uint32_t)v << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

}  // namespace

namespace orch_detail {
// error reporting for the host-only entry points of other translation units
int set_error(int code, const char* msg) { return fail(code, "%s", msg); }
}  // namespace orch_detail

struct orch_ctx {
  orch_dit_config cfg;
  int device = 0;
  int R = 0, n_kv = 0, H = 0, F = 0, L = 0, heads = 0, d = 0, B = 0, n_mod = 0, pdim = 0, odim = 0;
  bool loaded = false;

  // weights (T = config dtype unless noted)
  void* wbuf = nullptr;   // T matrices
  float* fbuf = nullptr;  // fp32 vectors and tables
  const void *w_t1 = nullptr, *w_t2 = nullptr, *table = nullptr, *w_ada = nullptr,
             *w_final = nullptr;
  std::vector<const void*> w_qkv, w_proj, w_fc1, w_fc2;
  const float *b_t1 = nullptr, *b_t2 = nullptr, *b_ada = nullptr, *b_final = nullptr,
              *w_pe = nullptr, *b_pe = nullptr, *pos = nullptr;
  std::vector<const float*> b_qkv, b_proj, b_fc1, b_fc2;

  // workspace, sized for a band of every row
  void* ws = nullptr;
  float* h = nullptr;
  void* u = nullptr;
  void* q = nullptr;
  void* kvf = nullptr;
  void* att = nullptr;
  void* mlp = nullptr;
  float* mod = nullptr;
  float* t1 = nullptr;
  float* sc = nullptr;
  float* eps = nullptr;
  void* attn_ws = nullptr;
  size_t attn_ws_bytes = 0;
  float* gemm_ws = nullptr;   // k-split partials of short (small-band) GEMMs
  size_t gemm_ws_elems = 0;
  float* lat[3] = {};   // latents of the patch-parallel sampler
  bool work_split = true;   // k-split of short GEMMs, cut attention query tiles

  // per-kernel timing: event pairs recorded around each launch of a step
  struct Timing {
    bool on = false;
    std::vector<hipEvent_t> ev;   // 2 per record
    std::vector<int> cls;
    size_t used = 0;
    double ms[ORCH_KCLASS_COUNT] = {};
    long long n[ORCH_KCLASS_COUNT] = {};
  } timing;
};

namespace {

int validate_config(const orch_dit_config* c) {
  if (!c) return fail(ORCH_EINVAL, "config is NULL");
  if (c->n_blocks < 1 || c->hidden < 1 || c->heads < 1 || c->mlp_hidden < 1)
    return fail(ORCH_EINVAL, "n_blocks, hidden, heads, mlp_hidden must be positive");
  if (c->hidden % c->heads) return fail(ORCH_EINVAL, "hidden %% heads != 0");
  const int d = c->hidden / c->heads;
  if (!(d == 32 || d == 64 || d == 72 || d == 80 || d == 96 || d == 128))
    return fail(ORCH_EINVAL, "head_dim %d not in {32,64,72,80,96,128}", d);
  if (c->hidden % 128 || c->hidden > 2048) return fail(ORCH_EINVAL, "hidden must be a multiple of 128, <= 2048");
  if (c->patch != 2) return fail(ORCH_EINVAL, "patch must be 2");
  if (c->in_ch * c->patch * c->patch != 16 || c->out_ch * c->patch * c->patch != 16)
    return fail(ORCH_EINVAL, "in_ch * patch^2 and out_ch * patch^2 must be 16");
  if (c->latent < c->patch || c->latent % c->patch) return fail(ORCH_EINVAL, "latent %% patch != 0");
  if (((c->latent / c->patch) * (c->latent / c->patch)) % 64)
    return fail(ORCH_EINVAL, "token count must be a multiple of 64");
  if (c->num_classes < 1 || c->freq_dim < 2 || c->freq_dim % 2)
    return fail(ORCH_EINVAL, "num_classes / freq_dim invalid");
  if (c->cfg_batch != 1 && c->cfg_batch != 2) return fail(ORCH_EINVAL, "cfg_batch must be 1 or 2");
  if (c->dtype != ORCH_F32 && c->dtype != ORCH_BF16) return fail(ORCH_EINVAL, "dtype must be F32 or BF16");
  if (c->T < 2 || !(c->beta_start > 0) || !(c->beta_end < 1) || c->beta_end < c->beta_start)
    return fail(ORCH_EINVAL, "schedule invalid");
  return ORCH_OK;
}

// alpha_bar of the linear-beta schedule; t < 0 -> 1.
double alpha_bar(const orch_dit_config& c, int t) {
  if (t < 0) return 1.0;
  double p = 1.0;
  for (int i = 0; i <= t; ++i) {
    const double beta = c.beta_start + (c.beta_end - c.beta_start) * (double)i / (double)(c.T - 1);
    p *= 1.0 - beta;
  }
  return p;
}

// x_prev = a x - b eps + c z for the step t -> t_prev (eta-DDIM; eta = 0 is
// the deterministic first-order update of Lemma 1, written so that the final
// step t_prev = -1 (sigma_prev = 0) stays finite).
void coefficients(const orch_dit_config& cfg, int t, int t_prev, double eta, double out[3]) {
  const double ab_s = alpha_bar(cfg, t), ab_p = alpha_bar(cfg, t_prev);
  const double a_s = std::sqrt(ab_s), s_s = std::sqrt(1.0 - ab_s), a_p = std::sqrt(ab_p);
  double c = 0.0;
  if (eta > 0.0) c = eta * std::sqrt((1.0 - ab_p) / (1.0 - ab_s)) * std::sqrt(1.0 - ab_s / ab_p);
  out[0] = a_p / a_s;
  out[1] = a_p * s_s / a_s - std::sqrt(std::fmax(0.0, 1.0 - ab_p - c * c));
  out[2] = c;
}

struct Tensor {
  size_t offset, count;
};

// Tensor table of the blob, in blob order (must mirror the documented format).
std::vector<Tensor> blob_table(const orch_ctx& x, size_t* total) {
  std::vector<Tensor> t;
  size_t off = 256;
  const size_t es = esize(x.cfg.dtype);
  auto add = [&](size_t n) {
    t.push_back({off, n});
    off = (off + n * es + 255) / 256 * 256;
  };
  const size_t H = x.H, F = x.F;
  add(H * x.pdim); add(H);                         // x_embedder
  add((size_t)x.n_kv * H);                          // pos_embed
  add(H * x.cfg.freq_dim); add(H);                  // t_embedder.fc1
  add(H * H); add(H);                               // t_embedder.fc2
  add((size_t)(x.cfg.num_classes + 1) * H);         // y_embedder.table
  for (int l = 0; l < x.L; ++l) {
    add(6 * H * H); add(6 * H);
    add(3 * H * H); add(3 * H);
    add(H * H); add(H);
    add(F * H); add(F);
    add(H * F); add(H);
  }
  add(2 * H * H); add(2 * H);
  add((size_t)x.odim * H); add(x.odim);
  *total = off;
  return t;
}

}  // namespace

extern "C" {

const char* orch_last_error(void) { return g_err.c_str(); }

int orch_schedule_coefficients(const orch_dit_config* cfg, int t, int t_prev, double eta,
                               double out_abc[3]) {
  if (!cfg || !out_abc) return fail(ORCH_EINVAL, "NULL argument");
  if (cfg->T < 2 || t < 0 || t >= cfg->T || t_prev < -1 || t_prev >= t)
    return fail(ORCH_EINVAL, "need 0 <= t < T and -1 <= t_prev < t (t=%d, t_prev=%d)", t, t_prev);
  if (!(eta >= 0.0)) return fail(ORCH_EINVAL, "eta must be >= 0");
  coefficients(*cfg, t, t_prev, eta, out_abc);
  return ORCH_OK;
}

int orch_create(const orch_dit_config* cfg, orch_ctx** out) {
  if (!out) return fail(ORCH_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = validate_config(cfg);
  if (rc) return rc;
  orch_ctx* x = new orch_ctx();
  x->cfg = *cfg;
  HIP_TRY(hipGetDevice(&x->device), "hipGetDevice");
  x->H = cfg->hidden;
  x->F = cfg->mlp_hidden;
  x->L = cfg->n_blocks;
  x->heads = cfg->heads;
  x->d = cfg->hidden / cfg->heads;
  x->B = cfg->cfg_batch;
  x->R = cfg->latent / cfg->patch;
  x->n_kv = x->R * x->R;
  x->n_mod = 6 * x->H * x->L + 2 * x->H;
  x->pdim = cfg->in_ch * cfg->patch * cfg->patch;
  x->odim = cfg->out_ch * cfg->patch * cfg->patch;

  const size_t es = esize(cfg->dtype);
  const size_t tokB = (size_t)x->B * x->n_kv;
  struct Part { size_t bytes; void** dst; };
  void *p_h, *p_u, *p_q, *p_kvf, *p_att, *p_mlp, *p_mod, *p_t1, *p_sc, *p_eps, *p_aws, *p_gws;
  void* p_lat[3];
  const size_t lat_bytes = (size_t)cfg->in_ch * cfg->latent * cfg->latent * 4;
  // split-KV partials: the largest need over every band height
  size_t aws = 0;
  for (int r = 1; r <= x->R; ++r)
    aws = std::max(aws, attention_workspace_bytes(x->B, x->heads, r * x->R, x->n_kv, x->d, cfg->dtype));
  x->attn_ws_bytes = aws;
  // GEMM k-split partials: the largest need over every band height and the
  // four projections
  size_t gws = 0;
  for (int r = 1; r <= x->R; ++r) {
    const int M = x->B * r * x->R;
    gws = std::max({gws, gemm_split_workspace_elems(M, 3 * x->H, x->H, cfg->dtype),
                    gemm_split_workspace_elems(M, x->H, x->H, cfg->dtype),
                    gemm_split_workspace_elems(M, x->F, x->H, cfg->dtype),
                    gemm_split_workspace_elems(M, x->H, x->F, cfg->dtype)});
  }
  x->gemm_ws_elems = gws;
  const Part parts[] = {
      {tokB * x->H * 4, &p_h},        {tokB * x->H * es, &p_u},
      {tokB * x->H * es, &p_q},       {2 * tokB * x->H * es, &p_kvf},
      {tokB * x->H * es, &p_att},     {tokB * x->F * es, &p_mlp},
      {(size_t)x->B * x->n_mod * 4, &p_mod}, {(size_t)x->H * 4, &p_t1},
      {(size_t)x->B * x->H * 4, &p_sc},
      {(size_t)x->B * cfg->out_ch * cfg->latent * cfg->latent * 4, &p_eps},
      {aws, &p_aws}, {lat_bytes, &p_lat[0]}, {lat_bytes, &p_lat[1]}, {lat_bytes, &p_lat[2]},
      {gws * 4, &p_gws}};
  size_t total = 0;
  for (const Part& p : parts) total += (p.bytes + 255) / 256 * 256;
  hipError_t e = hipMalloc(&x->ws, total);
  if (e != hipSuccess) {
    delete x;
    return fail(ORCH_ENOMEM, "workspace hipMalloc(%zu): %s", total, hipGetErrorString(e));
  }
  size_t off = 0;
  for (const Part& p : parts) {
    *p.dst = (char*)x->ws + off;
    off += (p.bytes + 255) / 256 * 256;
  }
  x->h = (float*)p_h; x->u = p_u; x->q = p_q; x->kvf = p_kvf; x->att = p_att; x->mlp = p_mlp;
  x->mod = (float*)p_mod; x->t1 = (float*)p_t1; x->sc = (float*)p_sc; x->eps = (float*)p_eps;
  x->attn_ws = aws ? p_aws : nullptr;
  x->gemm_ws = gws ? (float*)p_gws : nullptr;
  for (int i = 0; i < 3; ++i) x->lat[i] = (float*)p_lat[i];
  *out = x;
  return ORCH_OK;
}

void orch_destroy(orch_ctx* x) {
  if (!x) return;
  for (hipEvent_t e : x->timing.ev) (void)hipEventDestroy(e);
  if (x->ws) (void)hipFree(x->ws);
  if (x->wbuf) (void)hipFree(x->wbuf);
  if (x->fbuf) (void)hipFree(x->fbuf);
  delete x;
}

size_t orch_stale_kv_bytes(const orch_ctx* x) {
  if (!x) return 0;
  return (size_t)x->L * x->B * 2 * x->n_kv * x->H * esize(x->cfg.dtype);
}

int orch_load_dit_weights(orch_ctx* x, const void* host_blob, size_t nbytes) {
  if (!x || !host_blob) return fail(ORCH_EINVAL, "NULL argument");
  if (nbytes < 256) return fail(ORCH_EINVAL, "blob shorter than its header");
  const unsigned char* blob = (const unsigned char*)host_blob;
  if (memcmp(blob, "ORCHDIT1", 8) != 0) return fail(ORCH_EINVAL, "bad blob magic");
  uint32_t hv[13];
  memcpy(hv, blob + 8, sizeof hv);
  const orch_dit_config& c = x->cfg;
  const uint32_t want[13] = {1u, (uint32_t)c.dtype, (uint32_t)c.n_blocks, (uint32_t)c.hidden,
                             (uint32_t)c.heads, (uint32_t)c.mlp_hidden, (uint32_t)c.in_ch,
                             (uint32_t)c.out_ch, (uint32_t)c.patch, (uint32_t)x->R,
                             (uint32_t)c.num_classes, (uint32_t)c.freq_dim, 0u};
  static const char* names[13] = {"version", "dtype", "n_blocks", "hidden", "heads", "mlp_hidden",
                                  "in_ch", "out_ch", "patch", "grid", "num_classes", "freq_dim", ""};
  for (int i = 0; i < 12; ++i)
    if (hv[i] != want[i])
      return fail(ORCH_EINVAL, "blob header %s = %u, context expects %u", names[i], hv[i], want[i]);
  size_t total = 0;
  std::vector<Tensor> tab = blob_table(*x, &total);
  if (hv[12] != tab.size()) return fail(ORCH_EINVAL, "blob tensor count %u != %zu", hv[12], tab.size());
  if (nbytes < total) return fail(ORCH_EINVAL, "blob has %zu bytes, format needs %zu", nbytes, total);

  const size_t es = esize(c.dtype);
  auto to_f32 = [&](const Tensor& t, float* dst) {
    const unsigned char* src = blob + t.offset;
    if (c.dtype == ORCH_F32) {
      memcpy(dst, src, t.count * 4);
    } else {
      for (size_t i = 0; i < t.count; ++i) {
        uint16_t v;
        memcpy(&v, src + 2 * i, 2);
        dst[i] = bf16_bits_to_float(v);
      }
    }
  };

  // T matrices: t_embedder fc1, fc2, label table, adaLN (blocks then final,
  // concatenated into one [n_mod][H] matrix), per-block qkv/proj/fc1/fc2,
  // final linear.
  const size_t H = x->H, F = x->F;
  const int per_block = 10, first_block = 8;
  std::vector<std::pair<const Tensor*, size_t>> wlist;  // (tensor, dst offset in elements)
  size_t woff = 0;
  auto wadd = [&](const Tensor& t) {
    wlist.push_back({&t, woff});
    size_t at = woff;
    woff = (woff + t.count + 127) / 128 * 128;
    return at;
  };
  const size_t o_t1 = wadd(tab[3]);
  const size_t o_t2 = wadd(tab[5]);
  const size_t o_tab = wadd(tab[7]);
  // adaLN: the block matrices and the final one as one [n_mod][H] matrix,
  // held in the 64-row groups of the conditioning GEMV (copied below)
  const size_t o_ada = woff;
  const size_t nb_final = first_block + per_block * x->L;
  woff += (size_t)(x->n_mod + 63) / 64 * 64 * H;
  woff = (woff + 127) / 128 * 128;
  std::vector<size_t> o_qkv(x->L), o_proj(x->L), o_fc1(x->L), o_fc2(x->L);
  for (int l = 0; l < x->L; ++l) {
    const int base = first_block + per_block * l;
    o_qkv[l] = wadd(tab[base + 2]);
    o_proj[l] = wadd(tab[base + 4]);
    o_fc1[l] = wadd(tab[base + 6]);
    o_fc2[l] = wadd(tab[base + 8]);
  }
  const size_t o_final = wadd(tab[nb_final + 2]);
  std::vector<unsigned char> hw(woff * es);
  for (auto& pr : wlist) memcpy(hw.data() + pr.second * es, blob + pr.first->offset, pr.first->count * es);
  {
    // adaLN rows: block l's 6H rows, then the final 2H, each row H elements
    size_t row = 0;
    auto put = [&](const Tensor& t, size_t rows) {
      const unsigned char* src = blob + t.offset;
      const size_t ch = 16 / es;   // elements per 16-byte chunk, kept together
      for (size_t r = 0; r < rows; ++r, ++row)
        for (size_t c = 0; c < H; c += ch)
          memcpy(hw.data() + (o_ada + adaln_group_index(row, c, (int)H, (int)es)) * es,
                 src + (r * H + c) * es, 16);
    };
    for (int l = 0; l < x->L; ++l) put(tab[first_block + per_block * l + 0], 6 * H);
    put(tab[nb_final + 0], 2 * H);
  }

  // fp32 vectors: biases (adaLN concatenated), patch-embedding weight, position table.
  std::vector<float> hf;
  auto fadd = [&](const Tensor& t) {
    size_t at = hf.size();
    hf.resize(at + (t.count + 63) / 64 * 64);
    to_f32(t, hf.data() + at);
    return at;
  };
  // patch-embedding weight, stored transposed [C*p*p][H] for coalesced reads
  const size_t f_pe_w = hf.size();
  {
    std::vector<float> wpe(tab[0].count);
    to_f32(tab[0], wpe.data());
    hf.resize(f_pe_w + (tab[0].count + 63) / 64 * 64);
    for (size_t n = 0; n < H; ++n)
      for (int k = 0; k < x->pdim; ++k) hf[f_pe_w + (size_t)k * H + n] = wpe[n * x->pdim + k];
  }
  const size_t f_pe_b = fadd(tab[1]);
  const size_t f_pos = fadd(tab[2]);
  const size_t f_t1 = fadd(tab[4]);
  const size_t f_t2 = fadd(tab[6]);
  const size_t f_ada = hf.size();
  hf.resize(f_ada + (size_t)x->n_mod);
  for (int l = 0; l < x->L; ++l) to_f32(tab[first_block + per_block * l + 1], hf.data() + f_ada + 6 * H * l);
  to_f32(tab[nb_final + 1], hf.data() + f_ada + 6 * H * x->L);
  hf.resize((hf.size() + 63) / 64 * 64);
  std::vector<size_t> f_qkv(x->L), f_proj(x->L), f_fc1(x->L), f_fc2(x->L);
  for (int l = 0; l < x->L; ++l) {
    const int base = first_block + per_block * l;
    f_qkv[l] = fadd(tab[base + 3]);
    f_proj[l] = fadd(tab[base + 5]);
    f_fc1[l] = fadd(tab[base + 7]);
    f_fc2[l] = fadd(tab[base + 9]);
  }
  const size_t f_final = fadd(tab[nb_final + 3]);
  (void)F;

  if (x->wbuf) { (void)hipFree(x->wbuf); x->wbuf = nullptr; }
  if (x->fbuf) { (void)hipFree(x->fbuf); x->fbuf = nullptr; }
  x->loaded = false;
  hipError_t e = hipMalloc(&x->wbuf, hw.size());
  if (e != hipSuccess) return fail(ORCH_ENOMEM, "weights hipMalloc(%zu): %s", hw.size(), hipGetErrorString(e));
  e = hipMalloc((void**)&x->fbuf, hf.size() * 4);
  if (e != hipSuccess) return fail(ORCH_ENOMEM, "weights hipMalloc(%zu): %s", hf.size() * 4, hipGetErrorString(e));
  HIP_TRY(hipMemcpy(x->wbuf, hw.data(), hw.size(), hipMemcpyHostToDevice), "hipMemcpy weights");
  HIP_TRY(hipMemcpy(x->fbuf, hf.data(), hf.size() * 4, hipMemcpyHostToDevice), "hipMemcpy weights");

  auto W = [&](size_t o) -> const void* { return (const char*)x->wbuf + o * es; };
  auto Fp = [&](size_t o) -> const float* { return x->fbuf + o; };
  x->w_t1 = W(o_t1); x->w_t2 = W(o_t2); x->table = W(o_tab); x->w_ada = W(o_ada);
  x->w_final = W(o_final);
  x->w_qkv.resize(x->L); x->w_proj.resize(x->L); x->w_fc1.resize(x->L); x->w_fc2.resize(x->L);
  x->b_qkv.resize(x->L); x->b_proj.resize(x->L); x->b_fc1.resize(x->L); x->b_fc2.resize(x->L);
  for (int l = 0; l < x->L; ++l) {
    x->w_qkv[l] = W(o_qkv[l]); x->w_proj[l] = W(o_proj[l]);
    x->w_fc1[l] = W(o_fc1[l]); x->w_fc2[l] = W(o_fc2[l]);
    x->b_qkv[l] = Fp(f_qkv[l]); x->b_proj[l] = Fp(f_proj[l]);
    x->b_fc1[l] = Fp(f_fc1[l]); x->b_fc2[l] = Fp(f_fc2[l]);
  }
  x->w_pe = Fp(f_pe_w); x->b_pe = Fp(f_pe_b); x->pos = Fp(f_pos);
  x->b_t1 = Fp(f_t1); x->b_t2 = Fp(f_t2); x->b_ada = Fp(f_ada); x->b_final = Fp(f_final);
  x->loaded = true;
  return ORCH_OK;
}

}  // extern "C"

namespace {

int check_device(const orch_ctx* x) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev), "hipGetDevice");
  if (dev != x->device) return fail(ORCH_EINVAL, "current device %d is not the context's device %d", dev, x->device);
  hipError_t pending = hipGetLastError();
  if (pending != hipSuccess) return hip_fail(pending, "earlier asynchronous error");
  return ORCH_OK;
}

int check_labels(const orch_ctx* x, const int* labels) {
  if (!labels) return fail(ORCH_EINVAL, "labels is NULL");
  for (int b = 0; b < x->B; ++b)
    if (labels[b] < 0 || labels[b] > x->cfg.num_classes)
      return fail(ORCH_EINVAL, "label %d out of [0, %d]", labels[b], x->cfg.num_classes);
  return ORCH_OK;
}

constexpr size_t kTimingRecords = 8192;

// Fold the recorded event pairs into the per-class sums (synchronises).
int timing_flush(orch_ctx* x) {
  auto& T = x->timing;
  if (!T.used) return ORCH_OK;
  HIP_TRY(hipEventSynchronize(T.ev[2 * T.used - 1]), "hipEventSynchronize");
  for (size_t i = 0; i < T.used; ++i) {
    float ms = 0.0f;
    HIP_TRY(hipEventElapsedTime(&ms, T.ev[2 * i], T.ev[2 * i + 1]), "hipEventElapsedTime");
    T.ms[T.cls[i]] += ms;
    T.n[T.cls[i]] += 1;
  }
  T.used = 0;
  return ORCH_OK;
}

// Record the start / stop of one launch of class `c` (no-op when off).
struct KernelTimer {
  orch_ctx* x;
  hipStream_t s;
  int c;
  bool active = false;
  KernelTimer(orch_ctx* x_, int c_, hipStream_t s_) : x(x_), s(s_), c(c_) {
    auto& T = x->timing;
    if (!T.on) return;
    if (T.used == kTimingRecords && timing_flush(x) != ORCH_OK) return;
    if (hipEventRecord(T.ev[2 * T.used], s) != hipSuccess) return;
    active = true;
  }
  ~KernelTimer() {
    if (!active) return;
    auto& T = x->timing;
    if (hipEventRecord(T.ev[2 * T.used + 1], s) == hipSuccess) T.cls[T.used++] = c;
  }
};

int run_conditioning(orch_ctx* x, int t, const int* labels, float* mod, hipStream_t s) {
  CondParams cp{};
  cp.w_t1 = x->w_t1; cp.b_t1 = x->b_t1; cp.w_t2 = x->w_t2; cp.b_t2 = x->b_t2;
  cp.table = x->table; cp.w_ada = x->w_ada; cp.b_ada = x->b_ada;
  cp.hidden = x->H; cp.freq_dim = x->cfg.freq_dim; cp.n_mod = x->n_mod; cp.B = x->B;
  cp.labels[0] = labels[0];
  cp.labels[1] = x->B > 1 ? labels[1] : 0;
  cp.t = (float)t;
  cp.t1 = x->t1; cp.sc = x->sc; cp.mod = mod;
  KernelTimer kt(x, ORCH_KCLASS_CONDITIONING, s);
  HIP_TRY(launch_conditioning(cp, x->cfg.dtype, s), "conditioning launch");
  return ORCH_OK;
}

int run_patch_embed(orch_ctx* x, const float* x_full, int rb, int re, float* out, hipStream_t s) {
  PatchEmbedParams pp{};
  pp.x = x_full; pp.w = x->w_pe; pp.b = x->b_pe; pp.pos = x->pos; pp.h = out;
  pp.C = x->cfg.in_ch; pp.latent = x->cfg.latent; pp.patch = x->cfg.patch; pp.grid = x->R;
  pp.hidden = x->H; pp.row_begin = rb; pp.n_rows = re - rb; pp.B = x->B;
  KernelTimer kt(x, ORCH_KCLASS_PATCH_EMBED, s);
  HIP_TRY(launch_patch_embed(pp, s), "patch-embed launch");
  return ORCH_OK;
}

int run_final(orch_ctx* x, const float* h, int rb, int re, const float* mod, float* eps, hipStream_t s) {
  const int n_tok = (re - rb) * x->R;
  const int dt = x->cfg.dtype;
  const float* shift = mod + (size_t)6 * x->H * x->L;
  {
    KernelTimer kt(x, ORCH_KCLASS_LAYERNORM, s);
    HIP_TRY(launch_layernorm_modulate(h, x->B * n_tok, x->H, n_tok, shift, shift + x->H,
                                      x->n_mod, x->u, dt, s), "final LN launch");
  }
  FinalParams fp{};
  fp.u = x->u; fp.w = x->w_final; fp.b = x->b_final; fp.eps = eps;
  fp.B = x->B; fp.n_tok = n_tok; fp.hidden = x->H; fp.out_ch = x->cfg.out_ch;
  fp.patch = x->cfg.patch; fp.grid = x->R; fp.n_rows = re - rb;
  KernelTimer kt(x, ORCH_KCLASS_FINAL, s);
  HIP_TRY(launch_final_linear(fp, dt, s), "final linear launch");
  return ORCH_OK;
}

}  // namespace

extern "C" {

namespace {

// One executed step of one band, arguments already validated.  kv_in is
// read for the tokens outside the band.  The band's fresh K/V go to kv_out
// (buffer layout, band tokens only) when it is non-NULL -- kv_out == kv_in
// is the in-place refresh -- else to the workspace.  The band of x_{t_prev}
// is written at out_x, channel c at out_x + c * ldo.
int run_step(orch_ctx* x, const float* x_full, int rb, int re, int t, int t_prev,
             const int* labels, float cfg_scale, void* kv_in, void* kv_out, const float* z,
             float eta, float* out_eps, float* out_x, int ldo, hipStream_t s) {
  const orch_dit_config& c = x->cfg;
  const int p = c.patch;
  const int n_rows = re - rb;
  const int n_tok = n_rows * x->R;
  const size_t lat2 = (size_t)c.latent * c.latent;
  int rc;
  double abc[3];
  coefficients(c, t, t_prev, eta, abc);
  const int dt = c.dtype;
  const size_t es = esize(dt);
  const int H = x->H, F = x->F, B = x->B;
  const int M = B * n_tok;
  float* gemm_ws = x->work_split ? x->gemm_ws : nullptr;
  void* attn_ws = x->work_split ? x->attn_ws : nullptr;

  rc = run_conditioning(x, t, labels, x->mod, s);
  if (rc) return rc;
  rc = run_patch_embed(x, x_full, rb, re, x->h, s);
  if (rc) return rc;

  // K/V destination of the QKV epilogue: kv_out (band tokens only) when
  // given, else the fresh workspace read by attention.
  const size_t stale_bs = (size_t)2 * x->n_kv * H;
  const size_t fresh_bs = (size_t)2 * n_tok * H;
  for (int l = 0; l < x->L; ++l) {
    const float* mb = x->mod + (size_t)6 * H * l;  // shift1 scale1 gate1 shift2 scale2 gate2
    void* layer_kv = (char*)kv_in + (size_t)l * B * stale_bs * es;
    void* layer_out = kv_out ? (char*)kv_out + (size_t)l * B * stale_bs * es : nullptr;

    {
      KernelTimer kt(x, ORCH_KCLASS_LAYERNORM, s);
      HIP_TRY(launch_layernorm_modulate(x->h, M, H, n_tok, mb, mb + H, x->n_mod, x->u, dt, s), "LN1 launch");
    }

    // with the MFMA attention, Q leaves the QKV epilogue already multiplied
    // by log2(e)/sqrt(d) (before its one rounding to bf16)
    const bool q_scaled = dt == kBF16 && attention_uses_mfma(x->d, x->n_kv, dt);
    EpiParams eq{};
    eq.q_scale = q_scaled ? 1.4426950408889634f / sqrtf((float)x->d) : 1.0f;
    eq.bias = x->b_qkv[l];
    eq.ws = gemm_ws; eq.ws_elems = x->gemm_ws_elems;
    eq.rows_per_batch = n_tok;
    eq.q = x->q;
    eq.heads = x->heads; eq.hidden = H; eq.head_dim = x->d;
    if (layer_out) {
      eq.kv = layer_out; eq.kv_branch_stride = stale_bs; eq.kv_tokens = x->n_kv; eq.tok_offset = rb * x->R;
    } else {
      eq.kv = x->kvf; eq.kv_branch_stride = fresh_bs; eq.kv_tokens = n_tok; eq.tok_offset = 0;
    }
    {
      KernelTimer kt(x, ORCH_KCLASS_QKV, s);
      HIP_TRY(launch_gemm(x->u, x->w_qkv[l], M, 3 * H, H, kEpiQkv, eq, dt, s), "QKV launch");
    }

    AttnParams ap{};
    ap.q = x->q; ap.kv_stale = layer_kv; ap.stale_bs = stale_bs;
    if (layer_out == layer_kv) {        // refreshed in place: every key in one buffer
      ap.kv_fresh = nullptr; ap.fresh_bs = 0; ap.fresh_begin = 0; ap.n_fresh = 0;
      ap.fresh_n = 0; ap.fresh_off = 0;
    } else if (layer_out) {             // band keys in kv_out, at their own tokens
      ap.kv_fresh = layer_out; ap.fresh_bs = stale_bs; ap.fresh_begin = rb * x->R;
      ap.n_fresh = n_tok; ap.fresh_n = x->n_kv; ap.fresh_off = rb * x->R;
    } else {                            // band keys in the compact workspace
      ap.kv_fresh = x->kvf; ap.fresh_bs = fresh_bs; ap.fresh_begin = rb * x->R;
      ap.n_fresh = n_tok; ap.fresh_n = n_tok; ap.fresh_off = 0;
    }
    ap.B = B; ap.heads = x->heads; ap.n_q = n_tok; ap.n_kv = x->n_kv; ap.d = x->d; ap.out = x->att;
    ap.q_scaled = q_scaled;
    ap.ws = attn_ws; ap.ws_bytes = x->attn_ws_bytes;
    {
      KernelTimer kt(x, ORCH_KCLASS_ATTENTION, s);
      HIP_TRY(launch_attention(ap, dt, s), "attention launch");
    }

    EpiParams eo{};
    eo.out = x->h; eo.bias = x->b_proj[l]; eo.gate = mb + 2 * H; eo.gate_stride = x->n_mod;
    eo.rows_per_batch = n_tok;
    eo.ws = gemm_ws; eo.ws_elems = x->gemm_ws_elems;
    {
      KernelTimer kt(x, ORCH_KCLASS_PROJ, s);
      HIP_TRY(launch_gemm(x->att, x->w_proj[l], M, H, H, kEpiResidual, eo, dt, s), "proj launch");
    }

    {
      KernelTimer kt(x, ORCH_KCLASS_LAYERNORM, s);
      HIP_TRY(launch_layernorm_modulate(x->h, M, H, n_tok, mb + 3 * H, mb + 4 * H, x->n_mod, x->u, dt, s), "LN2 launch");
    }

    EpiParams e1{};
    e1.out = x->mlp; e1.bias = x->b_fc1[l];
    e1.ws = gemm_ws; e1.ws_elems = x->gemm_ws_elems;
    {
      KernelTimer kt(x, ORCH_KCLASS_FC1, s);
      HIP_TRY(launch_gemm(x->u, x->w_fc1[l], M, F, H, kEpiGelu, e1, dt, s), "fc1 launch");
    }

    EpiParams e2{};
    e2.out = x->h; e2.bias = x->b_fc2[l]; e2.gate = mb + 5 * H; e2.gate_stride = x->n_mod;
    e2.rows_per_batch = n_tok;
    e2.ws = gemm_ws; e2.ws_elems = x->gemm_ws_elems;
    {
      KernelTimer kt(x, ORCH_KCLASS_FC2, s);
      HIP_TRY(launch_gemm(x->mlp, x->w_fc2[l], M, H, F, kEpiResidual, e2, dt, s), "fc2 launch");
    }
  }

  float* eps = out_eps ? out_eps : x->eps;
  rc = run_final(x, x->h, rb, re, x->mod, eps, s);
  if (rc) return rc;

  const size_t band_cols = (size_t)n_rows * p * c.latent;
  const float* xb = x_full + (size_t)rb * p * c.latent;
  const float* zb = z ? z + (size_t)rb * p * c.latent : nullptr;
  const float* ec = eps;
  const float* eu = B > 1 ? eps + (size_t)c.out_ch * band_cols : nullptr;
  {
    KernelTimer kt(x, ORCH_KCLASS_UPDATE, s);
    HIP_TRY(launch_update(xb, (int)lat2, ec, eu, cfg_scale, abc[2] != 0.0 ? zb : nullptr, (int)lat2,
                          (float)abc[0], (float)abc[1], (float)abc[2], out_x, ldo, c.in_ch,
                          band_cols, s),
            "update launch");
  }
  return ORCH_OK;
}

}  // namespace

int orch_patch_denoise_step(orch_ctx* x, const float* x_full, int rb, int re, int t, int t_prev,
                            const int* labels, float cfg_scale, void* stale_kv, int refresh,
                            const float* z, float eta, float* out_eps, float* out_x_patch,
                            void* hip_stream) {
  if (!x) return fail(ORCH_EINVAL, "ctx is NULL");
  if (!x->loaded) return fail(ORCH_ENOWEIGHTS, "weights not loaded");
  if (!x_full || !stale_kv || !out_x_patch) return fail(ORCH_EINVAL, "x_full, stale_kv and out_x_patch must be non-NULL");
  if (rb < 0 || re <= rb || re > x->R) return fail(ORCH_EINVAL, "band [%d, %d) not within [0, %d)", rb, re, x->R);
  if (t < 0 || t >= x->cfg.T || t_prev < -1 || t_prev >= t)
    return fail(ORCH_EINVAL, "need 0 <= t < T and -1 <= t_prev < t (t=%d, t_prev=%d)", t, t_prev);
  if (!(eta >= 0.0f) || !std::isfinite(eta)) return fail(ORCH_EINVAL, "eta must be finite and >= 0");
  if (eta > 0.0f && !z) return fail(ORCH_EINVAL, "eta > 0 needs z");
  if (!std::isfinite(cfg_scale)) return fail(ORCH_EINVAL, "cfg_scale must be finite");
  int rc = check_labels(x, labels);
  if (rc) return rc;
  const orch_dit_config& c = x->cfg;
  const int p = c.patch;
  const int n_rows = re - rb;
  const size_t lat2 = (size_t)c.latent * c.latent;
  const size_t x_bytes = c.in_ch * lat2 * 4;
  const size_t out_bytes = (size_t)c.in_ch * n_rows * p * c.latent * 4;
  const size_t eps_bytes = (size_t)x->B * c.out_ch * n_rows * p * c.latent * 4;
  const size_t kv_bytes = orch_stale_kv_bytes(x);
  // out_x_patch may be the band of x_full itself: the band is then updated in
  // place, in x_full's layout (channel stride latent * latent); any other
  // overlap with an input is an error
  const bool in_place = out_x_patch == x_full + (size_t)rb * p * c.latent;
  const size_t out_span = in_place ? x_bytes - (size_t)rb * p * c.latent * 4 : out_bytes;
  if ((!in_place && ranges_overlap(out_x_patch, out_bytes, x_full, x_bytes)) ||
      ranges_overlap(out_x_patch, out_span, stale_kv, kv_bytes) ||
      ranges_overlap(out_x_patch, out_span, out_eps, eps_bytes) ||
      ranges_overlap(out_eps, eps_bytes, x_full, x_bytes) ||
      ranges_overlap(out_eps, eps_bytes, stale_kv, kv_bytes))
    return fail(ORCH_EINVAL, "output buffers overlap inputs (out_x_patch may only be exactly the band of x_full)");
  if (((uintptr_t)x_full | (uintptr_t)stale_kv | (uintptr_t)out_x_patch | (uintptr_t)out_eps |
       (uintptr_t)z) & 15)
    return fail(ORCH_EINVAL, "device buffers must be 16-byte aligned");
  rc = check_device(x);
  if (rc) return rc;

  return run_step(x, x_full, rb, re, t, t_prev, labels, cfg_scale, stale_kv,
                  refresh ? stale_kv : nullptr, z, eta, out_eps, out_x_patch,
                  in_place ? (int)lat2 : n_rows * p * c.latent, (hipStream_t)hip_stream);
}

int orch_sample_patch_parallel(orch_ctx* x, float* latent, int n_bands, const int* row_splits,
                                const int* tiers, const int* t_grid, int steps, int warmup,
                                const int* labels, float cfg_scale, void* kv_a, void* kv_b,
                                void* hip_stream) {
  if (!x) return fail(ORCH_EINVAL, "ctx is NULL");
  if (!x->loaded) return fail(ORCH_ENOWEIGHTS, "weights not loaded");
  if (!latent || !row_splits || !tiers || !t_grid || !kv_a || !kv_b)
    return fail(ORCH_EINVAL, "NULL argument");
  if (n_bands < 1) return fail(ORCH_EINVAL, "need n_bands >= 1");
  if (row_splits[0] != 0 || row_splits[n_bands] != x->R)
    return fail(ORCH_EINVAL, "row_splits must run from 0 to %d", x->R);
  for (int i = 0; i < n_bands; ++i) {
    if (row_splits[i + 1] <= row_splits[i]) return fail(ORCH_EINVAL, "row_splits must increase");
    if (tiers[i] != 0 && tiers[i] != 1) return fail(ORCH_EINVAL, "tiers must be 0 or 1");
  }
  if (steps < 1 || warmup < 1 || warmup > steps)
    return fail(ORCH_EINVAL, "need steps >= 1 and 1 <= warmup <= steps");
  if (t_grid[steps] != -1) return fail(ORCH_EINVAL, "t_grid[steps] must be -1");
  for (int m = 0; m < steps; ++m)
    if (t_grid[m] >= x->cfg.T || t_grid[m] <= t_grid[m + 1])
      return fail(ORCH_EINVAL, "t_grid must decrease from below T to -1");
  if (!std::isfinite(cfg_scale)) return fail(ORCH_EINVAL, "cfg_scale must be finite");
  int rc = check_labels(x, labels);
  if (rc) return rc;
  const orch_dit_config& c = x->cfg;
  const size_t lat2 = (size_t)c.latent * c.latent;
  const size_t lat_bytes = c.in_ch * lat2 * 4;
  const size_t kv_bytes = orch_stale_kv_bytes(x);
  if (ranges_overlap(kv_a, kv_bytes, kv_b, kv_bytes) ||
      ranges_overlap(latent, lat_bytes, kv_a, kv_bytes) ||
      ranges_overlap(latent, lat_bytes, kv_b, kv_bytes))
    return fail(ORCH_EINVAL, "latent and the two K/V buffers must not overlap");
  if (((uintptr_t)latent | (uintptr_t)kv_a | (uintptr_t)kv_b) & 15)
    return fail(ORCH_EINVAL, "device buffers must be 16-byte aligned");
  rc = check_device(x);
  if (rc) return rc;

  hipStream_t s = (hipStream_t)hip_stream;
  const int p = c.patch;
  float* xc = x->lat[0];   // latent at the current grid point
  float* xm = x->lat[1];   // a full-tier band after its first half-step
  float* xn = x->lat[2];   // latent at the interval's end
  void* bc = kv_a;         // buffer as of the last exchange
  void* bn = kv_b;         // exchanged K/V of the running interval
  HIP_TRY(hipMemcpyAsync(xc, latent, lat_bytes, hipMemcpyDeviceToDevice, s), "latent copy");
  // warm-up: synchronous exchange inside the step = the full-image step; the
  // buffer then holds that step's K/V of every token
  for (int m = 0; m < warmup; ++m) {
    rc = run_step(x, xc, 0, x->R, t_grid[m], t_grid[m + 1], labels, cfg_scale, bc, bc, nullptr,
                  0.0f, nullptr, xn, (int)lat2, s);
    if (rc) return rc;
    std::swap(xc, xn);
  }
  // sync intervals of two grid steps (one if a single step is left): every
  // device reads the buffer of the interval's start; a full-tier device
  // exchanges its first half-step's K/V and keeps its second's, a
  // reduced-tier device takes the double step and exchanges its K/V
  for (int m = warmup; m < steps;) {
    const int m2 = std::min(m + 2, steps);
    for (int i = 0; i < n_bands; ++i) {
      const int rb = row_splits[i], re = row_splits[i + 1];
      const size_t off = (size_t)rb * p * c.latent;
      if (tiers[i] == 0 && m2 == m + 2) {
        rc = run_step(x, xc, rb, re, t_grid[m], t_grid[m + 1], labels, cfg_scale, bc, bn,
                      nullptr, 0.0f, nullptr, xm + off, (int)lat2, s);
        if (rc) return rc;
        rc = run_step(x, xm, rb, re, t_grid[m + 1], t_grid[m + 2], labels, cfg_scale, bc,
                      nullptr, nullptr, 0.0f, nullptr, xn + off, (int)lat2, s);
      } else {
        rc = run_step(x, xc, rb, re, t_grid[m], t_grid[m2], labels, cfg_scale, bc, bn, nullptr,
                      0.0f, nullptr, xn + off, (int)lat2, s);
      }
      if (rc) return rc;
    }
    std::swap(xc, xn);
    std::swap(bc, bn);
    m = m2;
  }
  HIP_TRY(hipMemcpyAsync(latent, xc, lat_bytes, hipMemcpyDeviceToDevice, s), "latent copy");
  return ORCH_OK;
}

int orch_scheduler_update(const float* xin, const float* eps_cond, const float* eps_uncond,
                          float cfg_scale, const float* z, double a, double b, double c, float* out,
                          size_t n, void* hip_stream) {
  if (!xin || !eps_cond || !out) return fail(ORCH_EINVAL, "x, eps_cond and out must be non-NULL");
  if (c != 0.0 && !z) return fail(ORCH_EINVAL, "c != 0 needs z");
  if (!std::isfinite(a) || !std::isfinite(b) || !std::isfinite(c) || !std::isfinite(cfg_scale))
    return fail(ORCH_EINVAL, "coefficients must be finite");
  if (n == 0) return ORCH_OK;
  if (n > (size_t)1 << 40) return fail(ORCH_EINVAL, "n too large");
  hipError_t pending = hipGetLastError();
  if (pending != hipSuccess) return hip_fail(pending, "earlier asynchronous error");
  HIP_TRY(launch_update(xin, 0, eps_cond, eps_uncond, cfg_scale, c != 0.0 ? z : nullptr, 0, (float)a,
                        (float)b, (float)c, out, 0, 1, n, (hipStream_t)hip_stream),
          "update launch");
  return ORCH_OK;
}

// ---- kernel-level entry points -------------------------------------------

int orch_op_layernorm_modulate(const float* xin, int rows, int hidden, int rpb, const float* shift,
                               const float* scale, int mod_stride, void* out, int dtype,
                               void* hip_stream) {
  if (!xin || !shift || !scale || !out) return fail(ORCH_EINVAL, "NULL pointer");
  if (rows < 0 || rpb < 1 || hidden % 128 || hidden < 128 || hidden > 2048 || mod_stride < hidden)
    return fail(ORCH_EINVAL, "bad shape (hidden must be a multiple of 128, <= 2048)");
  if (dtype != ORCH_F32 && dtype != ORCH_BF16) return fail(ORCH_EINVAL, "bad dtype");
  HIP_TRY(launch_layernorm_modulate(xin, rows, hidden, rpb, shift, scale, mod_stride, out, dtype,
                                    (hipStream_t)hip_stream), "LN launch");
  return ORCH_OK;
}

size_t orch_linear_workspace_bytes(int M, int N, int K, int dtype) {
  if (dtype != ORCH_BF16 || M < 1 || N < 1 || K < 1) return 0;
  return gemm_split_workspace_elems(M, N, K, dtype) * sizeof(float);
}

int orch_op_linear(const void* A, int M, int K, const void* W, int N, const float* bias,
                   int epilogue, const float* gate, int gate_stride, int rpb, void* out,
                   void* workspace, size_t workspace_bytes, int dtype, void* hip_stream) {
  if (!A || !W || !bias || !out) return fail(ORCH_EINVAL, "NULL pointer");
  if (M < 0 || K < 1 || N < 1) return fail(ORCH_EINVAL, "bad shape");
  if (dtype != ORCH_F32 && dtype != ORCH_BF16) return fail(ORCH_EINVAL, "bad dtype");
  if (dtype == ORCH_BF16 && K % 8) return fail(ORCH_EINVAL, "bf16 needs K %% 8 == 0");
  if (epilogue != ORCH_EPI_STORE && epilogue != ORCH_EPI_GELU && epilogue != ORCH_EPI_RESIDUAL)
    return fail(ORCH_EINVAL, "bad epilogue");
  if (epilogue == ORCH_EPI_RESIDUAL && (!gate || rpb < 1 || gate_stride < N))
    return fail(ORCH_EINVAL, "residual epilogue needs gate, gate_stride >= N, rows_per_batch >= 1");
  EpiParams ep{};
  ep.out = out; ep.bias = bias; ep.gate = gate; ep.gate_stride = gate_stride;
  ep.rows_per_batch = rpb < 1 ? 1 : rpb;
  if (workspace) {
    ep.ws = (float*)workspace;
    ep.ws_elems = workspace_bytes / sizeof(float);
  }
  HIP_TRY(launch_gemm(A, W, M, N, K, epilogue, ep, dtype, (hipStream_t)hip_stream), "linear launch");
  return ORCH_OK;
}

int orch_op_qkv_projection(const void* A, int B, int n_tok, int K, const void* W, const float* bias,
                           int hidden, int heads, void* q_out, void* kv_out,
                           size_t kv_branch_stride, int kv_tokens, int tok_offset, int dtype,
                           void* hip_stream) {
  if (!A || !W || !bias || !q_out || !kv_out) return fail(ORCH_EINVAL, "NULL pointer");
  if (B < 1 || n_tok < 0 || K < 1 || heads < 1 || hidden % heads || tok_offset < 0 ||
      tok_offset + n_tok > kv_tokens || kv_branch_stride < (size_t)2 * kv_tokens * hidden)
    return fail(ORCH_EINVAL, "bad shape");
  if (dtype != ORCH_F32 && dtype != ORCH_BF16) return fail(ORCH_EINVAL, "bad dtype");
  if (dtype == ORCH_BF16 && K % 8) return fail(ORCH_EINVAL, "bf16 needs K %% 8 == 0");
  EpiParams ep{};
  ep.bias = bias; ep.rows_per_batch = n_tok < 1 ? 1 : n_tok; ep.q = q_out; ep.kv = kv_out;
  ep.kv_branch_stride = kv_branch_stride; ep.kv_tokens = kv_tokens; ep.tok_offset = tok_offset;
  ep.heads = heads; ep.hidden = hidden; ep.head_dim = hidden / heads;
  HIP_TRY(launch_gemm(A, W, B * n_tok, 3 * hidden, K, kEpiQkv, ep, dtype, (hipStream_t)hip_stream),
          "qkv launch");
  return ORCH_OK;
}

size_t orch_attention_workspace_bytes(int B, int heads, int n_q, int n_kv, int head_dim,
                                      int dtype) {
  if (B < 1 || heads < 1 || n_q < 0 || n_kv < 1 || head_dim < 1) return 0;
  return attention_workspace_bytes(B, heads, n_q, n_kv, head_dim, dtype);
}

}  // extern "C"

namespace orch_detail {

// Shape and pointer checks shared by the attention entry points.
int check_attention_args(const void* q, const void* kv_stale, size_t stale_bs,
                         const void* kv_fresh, size_t fresh_bs, int fresh_begin, int n_fresh,
                         int B, int heads, int n_q, int n_kv, int head_dim, const void* out,
                         int dtype) {
  if (!q || !kv_stale || !out || (n_fresh > 0 && !kv_fresh)) return fail(ORCH_EINVAL, "NULL pointer");
  if (B < 1 || heads < 1 || n_q < 0 || n_kv < 1 || n_fresh < 0 || fresh_begin < 0 ||
      fresh_begin + n_fresh > n_kv)
    return fail(ORCH_EINVAL, "bad shape");
  if (!(head_dim == 32 || head_dim == 64 || head_dim == 72 || head_dim == 80 || head_dim == 96 ||
        head_dim == 128))
    return fail(ORCH_EINVAL, "head_dim not supported");
  const size_t H = (size_t)heads * head_dim;
  if (stale_bs < 2 * (size_t)n_kv * H || (n_fresh > 0 && fresh_bs < 2 * (size_t)n_fresh * H))
    return fail(ORCH_EINVAL, "branch stride too small");
  if (dtype != ORCH_F32 && dtype != ORCH_BF16) return fail(ORCH_EINVAL, "bad dtype");
  return ORCH_OK;
}

AttnParams attention_params(const void* q, const void* kv_stale, size_t stale_bs,
                            const void* kv_fresh, size_t fresh_bs, int fresh_begin, int n_fresh,
                            int B, int heads, int n_q, int n_kv, int head_dim, void* out) {
  AttnParams ap{};
  ap.q = q; ap.kv_stale = kv_stale; ap.stale_bs = stale_bs; ap.kv_fresh = kv_fresh;
  ap.fresh_bs = fresh_bs; ap.fresh_begin = fresh_begin; ap.n_fresh = n_fresh; ap.B = B;
  ap.heads = heads; ap.n_q = n_q; ap.n_kv = n_kv; ap.d = head_dim; ap.out = out;
  ap.fresh_n = n_fresh; ap.fresh_off = 0;
  return ap;
}

}  // namespace orch_detail

extern "C" {

int orch_op_attention(const void* q, const void* kv_stale, size_t stale_bs, const void* kv_fresh,
                      size_t fresh_bs, int fresh_begin, int n_fresh, int B, int heads, int n_q,
                      int n_kv, int head_dim, void* out, void* workspace, size_t workspace_bytes,
                      int dtype, void* hip_stream) {
  int rc = orch_detail::check_attention_args(q, kv_stale, stale_bs, kv_fresh, fresh_bs,
                                             fresh_begin, n_fresh, B, heads, n_q, n_kv, head_dim,
                                             out, dtype);
  if (rc) return rc;
  AttnParams ap = orch_detail::attention_params(q, kv_stale, stale_bs, kv_fresh, fresh_bs, fresh_begin,
                                   n_fresh, B, heads, n_q, n_kv, head_dim, out);
  ap.ws = workspace; ap.ws_bytes = workspace ? workspace_bytes : 0;
  HIP_TRY(launch_attention(ap, dtype, (hipStream_t)hip_stream), "attention launch");
  return ORCH_OK;
}

int orch_op_conditioning(orch_ctx* x, int t, const int* labels, float* out, void* hip_stream) {
  if (!x || !out) return fail(ORCH_EINVAL, "NULL pointer");
  if (!x->loaded) return fail(ORCH_ENOWEIGHTS, "weights not loaded");
  if (t < 0 || t >= x->cfg.T) return fail(ORCH_EINVAL, "t out of range");
  int rc = check_labels(x, labels);
  if (rc) return rc;
  rc = check_device(x);
  if (rc) return rc;
  return run_conditioning(x, t, labels, out, (hipStream_t)hip_stream);
}

int orch_op_patch_embed(orch_ctx* x, const float* x_full, int rb, int re, float* out, void* hip_stream) {
  if (!x || !x_full || !out) return fail(ORCH_EINVAL, "NULL pointer");
  if (!x->loaded) return fail(ORCH_ENOWEIGHTS, "weights not loaded");
  if (rb < 0 || re <= rb || re > x->R) return fail(ORCH_EINVAL, "bad band");
  int rc = check_device(x);
  if (rc) return rc;
  return run_patch_embed(x, x_full, rb, re, out, (hipStream_t)hip_stream);
}

int orch_op_final_layer(orch_ctx* x, const float* h, int rb, int re, const float* mod, float* out_eps,
                        void* hip_stream) {
  if (!x || !h || !mod || !out_eps) return fail(ORCH_EINVAL, "NULL pointer");
  if (!x->loaded) return fail(ORCH_ENOWEIGHTS, "weights not loaded");
  if (rb < 0 || re <= rb || re > x->R) return fail(ORCH_EINVAL, "bad band");
  int rc = check_device(x);
  if (rc) return rc;
  return run_final(x, h, rb, re, mod, out_eps, (hipStream_t)hip_stream);
}

namespace {
int check_unet_shape(const orch_unet_conv_shape* s) {
  if (!s) return fail(ORCH_EINVAL, "shape is NULL");
  if (s->height < 1 || s->width < 1) return fail(ORCH_EINVAL, "height and width must be >= 1");
  if (s->channels < 64 || s->channels % 64) return fail(ORCH_EINVAL, "channels must be a positive multiple of 64");
  if (s->groups < 1 || s->groups > 256 || s->channels % s->groups)
    return fail(ORCH_EINVAL, "groups must divide channels and be <= 256");
  if (s->out_channels < 64 || s->out_channels % 64) return fail(ORCH_EINVAL, "out_channels must be a positive multiple of 64");
  if (!(s->eps > 0.0f) || !std::isfinite(s->eps)) return fail(ORCH_EINVAL, "eps must be finite and > 0");
  if ((size_t)(s->height + 2) * (s->width + 2) * s->channels * 2 >= kUNetMaxTileBytes ||
      (size_t)s->out_channels * 9 * s->channels * 2 >= kUNetMaxTileBytes)
    return fail(ORCH_EINVAL, "map or weight too large (2 GiB or more in bf16)");
  return ORCH_OK;
}
}  // namespace

size_t orch_unet_conv_workspace_bytes(const orch_unet_conv_shape* s, int band_rows) {
  if (!s || band_rows < 1 || s->groups < 1 || s->channels < 1) return 0;
  return unet_conv_workspace_bytes(s->width, s->channels, s->groups, s->out_channels, band_rows);
}

int orch_unet_conv_band(const orch_unet_conv_shape* s, int rb, int re, const float* x_band,
                        const float* gamma, const float* beta, const void* weight,
                        const float* bias, void* stale_act, float* stale_sums, int refresh,
                        float* out, void* workspace, size_t workspace_bytes, void* hip_stream) {
  int rc = check_unet_shape(s);
  if (rc) return rc;
  if (rb < 0 || re <= rb || re > s->height)
    return fail(ORCH_EINVAL, "band [%d, %d) not within [0, %d)", rb, re, s->height);
  if (!x_band || !gamma || !beta || !weight || !bias || !out || !workspace)
    return fail(ORCH_EINVAL, "NULL pointer");
  const bool all_rows = rb == 0 && re == s->height;
  if ((!all_rows || refresh) && (!stale_act || !stale_sums))
    return fail(ORCH_EINVAL, "stale_act and stale_sums are needed unless the band is every row without refresh");
  const int rows = re - rb;
  const size_t need = unet_conv_workspace_bytes(s->width, s->channels, s->groups, s->out_channels, rows);
  if (workspace_bytes < need) return fail(ORCH_EINVAL, "workspace has %zu bytes, needs %zu", workspace_bytes, need);
  if (((uintptr_t)x_band | (uintptr_t)gamma | (uintptr_t)beta | (uintptr_t)weight | (uintptr_t)bias |
       (uintptr_t)stale_act | (uintptr_t)stale_sums | (uintptr_t)out | (uintptr_t)workspace) & 15)
    return fail(ORCH_EINVAL, "device buffers must be 16-byte aligned");
  const size_t out_bytes = (size_t)rows * s->width * s->out_channels * 4;
  const size_t x_bytes = (size_t)rows * s->width * s->channels * 4;
  const size_t act_bytes = (size_t)s->height * s->width * s->channels * 2;
  const size_t sums_bytes = (size_t)s->height * s->groups * 8;
  if (ranges_overlap(out, out_bytes, x_band, x_bytes) || ranges_overlap(out, out_bytes, stale_act, act_bytes) ||
      ranges_overlap(out, out_bytes, stale_sums, sums_bytes) || ranges_overlap(workspace, need, out, out_bytes) ||
      ranges_overlap(workspace, need, stale_act, act_bytes) || ranges_overlap(workspace, need, x_band, x_bytes))
    return fail(ORCH_EINVAL, "output or workspace overlaps an input");
  hipError_t pending = hipGetLastError();
  if (pending != hipSuccess) return hip_fail(pending, "earlier asynchronous error");
  UNetConvParams p{};
  p.x = x_band; p.gamma = gamma; p.beta = beta; p.weight = weight; p.bias = bias;
  p.stale_act = stale_act; p.stale_sums = stale_sums; p.out = out;
  p.H = s->height; p.W = s->width; p.C = s->channels; p.G = s->groups; p.C_out = s->out_channels;
  p.row_begin = rb; p.row_end = re; p.refresh = refresh ? 1 : 0; p.eps = s->eps;
  HIP_TRY(launch_unet_conv(p, workspace, (hipStream_t)hip_stream), "U-Net band launch");
  return ORCH_OK;
}

int orch_set_work_split(orch_ctx* x, int enable) {
  if (!x) return fail(ORCH_EINVAL, "ctx is NULL");
  x->work_split = enable != 0;
  return ORCH_OK;
}

int orch_set_kernel_timing(orch_ctx* x, int enable) {
  if (!x) return fail(ORCH_EINVAL, "ctx is NULL");
  auto& T = x->timing;
  if (enable && !T.on) {
    T.ev.assign(2 * kTimingRecords, nullptr);
    for (auto& e : T.ev) {
      hipError_t r = hipEventCreate(&e);
      if (r != hipSuccess) {
        for (hipEvent_t f : T.ev)
          if (f) (void)hipEventDestroy(f);
        T.ev.clear();
        return hip_fail(r, "hipEventCreate");
      }
    }
    T.cls.assign(kTimingRecords, 0);
    T.used = 0;
    for (int i = 0; i < ORCH_KCLASS_COUNT; ++i) { T.ms[i] = 0.0; T.n[i] = 0; }
    T.on = true;
  } else if (!enable && T.on) {
    int rc = timing_flush(x);
    for (hipEvent_t e : T.ev) (void)hipEventDestroy(e);
    T.ev.clear();
    T.cls.clear();
    T.on = false;
    if (rc) return rc;
  }
  return ORCH_OK;
}

int orch_kernel_times(orch_ctx* x, double* total_ms, long long* launches) {
  if (!x) return fail(ORCH_EINVAL, "ctx is NULL");
  auto& T = x->timing;
  int rc = timing_flush(x);
  if (rc) return rc;
  for (int i = 0; i < ORCH_KCLASS_COUNT; ++i) {
    if (total_ms) total_ms[i] = T.ms[i];
    if (launches) launches[i] = T.n[i];
    T.ms[i] = 0.0;
    T.n[i] = 0;
  }
  return ORCH_OK;
}

}  // extern "C"
