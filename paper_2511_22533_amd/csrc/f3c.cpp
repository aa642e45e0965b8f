// Host side of the f3c C ABI: argument validation, weight and state layout in
// caller-provided device memory, and the stream-ordered orchestration of one
// cached denoising step (Algorithm 1): select -> gather/embed -> modulation ->
// L blocks on the compacted set -> final projection -> merge/Euler/rotate.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>
#include <cstdlib>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/f3c.h"
#include "common.h"
#include "kernels.h"

using namespace f3c;

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

#define HIP_TRY(expr)                                                                  \
  do {                                                                                 \
    hipError_t e_ = (expr);                                                            \
    if (e_ != hipSuccess) return fail(F3C_EHIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Attention key-split partials per state. A launch splits only while its
// 128-query tiles x heads x splits stay within 256 workgroups, so the partials
// never exceed 256 x 128 rows of head_dim + 2 floats (8.25 MiB at 64); with
// less room the launch uses fewer splits.
constexpr size_t kAttnWsBytes = size_t(12) << 20;

struct Spec {
  std::string name;
  int64_t rows, cols;   // cols == 0 for vectors
  bool bias;
  size_t off = 0;       // byte offset in the weight buffer
  int64_t numel() const { return cols ? rows * cols : rows; }
};

}  // namespace

struct f3c_model {
  f3c_model_cfg cfg;
  int N, d, hd, dm, L, dc, Nc;
  size_t es;
  std::vector<Spec> specs;
  size_t wbytes = 0;
  char* wdev = nullptr;
  bool loaded = false;
  // group bases (bytes)
  size_t mod_w, mod_b, kv_w, kv_b;
  // Byte offsets of the other weights, resolved from their names once at
  // creation so that a step does no name lookups.
  struct Top { size_t in_w, in_b, pos, t1_w, t1_b, t2_w, t2_b, out_w, out_b; } top{};
  struct Block { size_t qkv_w, qkv_b, o_w, o_b, q_w, q_b, co_w, co_b, fc1_w, fc1_b, fc2_w, fc2_b; };
  std::vector<Block> blk;

  const void* w(size_t off) const { return wdev + off; }
  const float* b(size_t off) const { return reinterpret_cast<const float*>(wdev + off); }
};

struct Prof {
  std::vector<hipEvent_t> ev;       // start/stop pairs
  int64_t launches = 0;
  double flops = 0, bytes = 0;
};

struct f3c_state {
  f3c_model* m;
  int B;
  char* dev;
  size_t bytes;
  float* v[2];
  int cur = 0;
  float *h, *vact, *mod, *temb, *score;
  void *u, *qkv, *att, *qc, *hid, *cond_t, *kv;
  int32_t *idx, *pos;
  void* sel_ws = nullptr;       // selection: magnitude pairs and partial extremes
  float* ws = nullptr;          // attention key-split partials
  size_t ws_bytes = 0;
  bool guided = false;          // activations and condition K/V sized for two passes per sample
  std::vector<double> plan_t;   // times of the modulation plan, [i] at plan_mod + i * L * 6d
  float* plan_mod = nullptr;
  float* trace = nullptr;       // debug: residual stream after the embedding and after each block
  size_t trace_bytes = 0;
  float* sub_trace = nullptr;   // debug: pre-gate sublayer outputs of each block
  size_t sub_trace_bytes = 0;
  const int32_t* force_idx = nullptr;   // debug: the next step's active sets (teacher forcing)
  const float* last_mod = nullptr;      // modulation vectors the last step read
  bool last_selected = false;           // the last step wrote idx/pos (some sample cached)
  bool cond_set = false, uncond_set = false, record_scores = false;
  uint32_t prof_mask = 0;
  float omega = 0.7f;
  Segs last_act{};
  Prof prof[F3C_PROF_CLASSES];
  std::vector<hipEvent_t> pool;
};

namespace {

hipEvent_t take_event(f3c_state* s) {
  if (!s->pool.empty()) {
    hipEvent_t e = s->pool.back();
    s->pool.pop_back();
    return e;
  }
  // Timing only (no host data is published through these events): without
  // the system-scope fence, recording one costs no cache writeback before the
  // next kernel, which would otherwise be counted in the timed interval.
  hipEvent_t e = nullptr;
  if (hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return nullptr;
  return e;
}

// Times one call's kernels when profiling is on for its class: the launches
// inside the scope stamp the event pair at their own start and end (see
// LaunchTimer). A scope that launched nothing records both events in place.
struct Scope {
  f3c_state* s;
  int cls;
  hipStream_t st;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  LaunchTimer saved;
  Scope(f3c_state* s_, int cls_, hipStream_t st_, double flops, double bytes) : s(s_), cls(cls_), st(st_) {
    if (!(s->prof_mask >> cls & 1u)) return;
    e0 = take_event(s);
    e1 = take_event(s);
    if (!e0 || !e1) { e0 = e1 = nullptr; return; }
    s->prof[cls].ev.push_back(e0);
    s->prof[cls].ev.push_back(e1);
    s->prof[cls].launches += 1;
    s->prof[cls].flops += flops;
    s->prof[cls].bytes += bytes;
    LaunchTimer& t = launch_timer();
    saved = t;
    t = LaunchTimer{e0, e1, false};
  }
  ~Scope() {
    if (!e1) return;
    LaunchTimer& t = launch_timer();
    if (!t.used) {
      (void)hipEventRecord(e0, st);
      (void)hipEventRecord(e1, st);
    }
    t = saved;
  }
};

int validate_cfg(const f3c_model_cfg* c) {
  if (!c) return fail(F3C_EINVAL, "cfg is NULL");
  if (c->dtype != F3C_F32 && c->dtype != F3C_BF16) return fail(F3C_EINVAL, "dtype must be F3C_F32 or F3C_BF16");
  if (c->in_ch != 8) return fail(F3C_EINVAL, "in_ch must be 8 (got %d)", c->in_ch);
  if (c->grid < 1) return fail(F3C_EINVAL, "grid must be >= 1");
  const int64_t n = (int64_t)c->grid * c->grid * c->grid;
  if (n > F3C_MAX_TOKENS) return fail(F3C_EINVAL, "grid^3 = %lld exceeds %d tokens", (long long)n, F3C_MAX_TOKENS);
  if (c->heads < 1 || c->width % c->heads) return fail(F3C_EINVAL, "width must be a multiple of heads");
  const int hd = c->width / c->heads;
  if (hd != 32 && hd != 64) return fail(F3C_EINVAL, "head_dim must be 32 or 64 (got %d)", hd);
  if (c->width % 128 || c->width > 2048) return fail(F3C_EINVAL, "width must be a multiple of 128, <= 2048");
  if ((c->width / 64) & ((c->width / 64) - 1)) return fail(F3C_EINVAL, "width/64 must be a power of two");
  if (c->depth < 1 || c->depth > 256) return fail(F3C_EINVAL, "depth must be in 1..256");
  if (c->mlp_ratio < 1 || c->mlp_ratio > 8) return fail(F3C_EINVAL, "mlp_ratio must be in 1..8");
  if (c->cond_tokens < 1 || c->cond_tokens > 65536) return fail(F3C_EINVAL, "cond_tokens must be in 1..65536");
  if (c->cond_width < 64 || c->cond_width % 64) return fail(F3C_EINVAL, "cond_width must be a multiple of 64");
  return F3C_OK;
}

uint16_t f32_to_bf16_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;   // NaN
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

double block_flops(int B, double n, double d, double H, double nc, double dc, double dm) {
  const double mod = 5 * B * d + 2 * B * d * 6 * d;
  const double ln = 3 * 7 * B * n * d;
  const double sa = 2 * B * n * d * 3 * d + 2 * B * H * n * n * (d / H) + 5 * B * H * n * n +
                    2 * B * H * n * n * (d / H) + 2 * B * n * d * d;
  const double ca = 2 * B * n * d * d + 2 * B * nc * dc * 2 * d + 2 * B * H * n * nc * (d / H) + 5 * B * H * n * nc +
                    2 * B * H * n * nc * (d / H) + 2 * B * n * d * d;
  const double mlp = 2 * B * n * d * dm + 5 * B * n * dm + 2 * B * n * dm * d;
  return mod + ln + sa + ca + mlp;
}

int check_state(f3c_state* s) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (!s->m->loaded) return fail(F3C_ESTATE, "weights not loaded");
  return F3C_OK;
}

// One step of Algorithm 1. A guided step (guide) runs the transformer on two
// copies of the compacted active set, the conditional pass in segments 0..B-1
// and the unconditional one in segments B..2B-1 (same tokens, the second
// condition's K/V), and merges (1 + w) v_cond - w v_uncond in the Euler kernel.
int run_step(f3c_state* s, float* x, double t, double t_next, const int32_t* n_cache, bool guide, double w,
             hipStream_t st) {
  f3c_model* m = s->m;
  const int B = s->B, N = m->N, d = m->d, L = m->L, dt = m->cfg.dtype;
  const size_t es = m->es;
  Segs act{}, quota{};
  act.B = quota.B = B;
  bool any_cached = false;
  for (int b = 0; b < B; ++b) {
    const int c = n_cache ? n_cache[b] : 0;
    quota.off[b] = c;
    act.off[b + 1] = act.off[b] + (N - c);
    any_cached |= c > 0;
  }
  const int arows = act.off[B];              // active rows (one pass)
  // Segments of the transformer: the active set once, or twice on a guided step.
  const int P = guide ? 2 : 1;
  Segs tact{}, cond_segs{};
  tact.B = cond_segs.B = P * B;
  for (int g = 0; g < P * B; ++g) {
    const int b = g % B;
    tact.off[g + 1] = tact.off[g] + (act.off[b + 1] - act.off[b]);
    cond_segs.off[g + 1] = cond_segs.off[g] + m->Nc;
  }
  const int trows = tact.off[P * B];
  float* v_cache = s->v[s->cur];
  float* v_prev = s->v[1 - s->cur];
  const int32_t* idx = nullptr;
  const int32_t* pos = nullptr;

  const int32_t* forced = s->force_idx;
  s->force_idx = nullptr;                   // a step consumes the hook
  if (any_cached && forced) {
    HIP_TRY(launch_force_active(forced, act, N, s->idx, s->pos, st));
    idx = s->idx;
    pos = s->pos;
  } else if (any_cached) {
    const float w_a = s->omega, w_v = 1.0f - w_a;
    Scope sc(s, F3C_PROF_SELECT, st, 0, (double)B * N * (64 + 4) + arows * 4.0);
    HIP_TRY(launch_select(v_cache, v_prev, B, N, w_a, w_v, quota, act, s->idx, s->pos,
                          s->record_scores ? s->score : nullptr, s->sel_ws, st));
    idx = s->idx;
    pos = s->pos;
  }
  const float* mod = s->mod;
  int planned = -1;
  for (size_t i = 0; i < s->plan_t.size() && planned < 0; ++i)
    if (s->plan_t[i] == t) planned = (int)i;
  if (planned >= 0) {
    mod = s->plan_mod + (size_t)planned * 6 * L * d;
  } else {
    Scope sc(s, F3C_PROF_MOD, st, 0, (double)es * d * (256 + d + 6.0 * L * d));
    const char* mw = m->wdev;
    HIP_TRY(launch_gemv(dt, m->w(m->top.t1_w), m->b(m->top.t1_b), nullptr, t, GEMV_IN_TIMESTEP, 1, d, 256, s->temb, st));
    HIP_TRY(launch_gemv(dt, m->w(m->top.t2_w), m->b(m->top.t2_b), s->temb, 0.0, GEMV_IN_PLAIN, 0, d, d, s->temb + d, st));
    HIP_TRY(launch_gemv_t(dt, mw + m->mod_w, (const float*)(mw + m->mod_b), s->temb + d, 6 * L * d, d, s->mod, st));
  }
  if (arows > 0) {
    {
      Scope sc(s, F3C_PROF_EMBED, st, 0, arows * (32.0 + d * es + P * d * 4.0));
      HIP_TRY(launch_embed(dt, x, N, idx, act, m->w(m->top.in_w), m->b(m->top.in_b), m->w(m->top.pos), d, s->h, guide ? arows : 0,
                           st));
    }
    const int dm = m->dm;
    const int rows = trows;                    // the transformer's rows (both passes when guided)
    const double lnb = rows * (double)d * (4 + es);
    // Algorithmic bytes of the dense kernels (least data each must move):
    // projections read A and W and write the output (f32 residual read and
    // written); attention reads Q, K, V and writes O.
    const double r = rows, dd = d, E = (double)es;
    auto proj_bytes = [&](double n, double k, bool resid) { return (r * k + n * k) * E + r * n * (resid ? 8.0 : E); };
    double cond_rows = 0;
    for (int g = 0; g < P * B; ++g) cond_rows += (tact.off[g + 1] > tact.off[g]) ? m->Nc : 0;
    const size_t hslice = (size_t)rows * d;       // trace size checked by step_common
    if (s->trace) HIP_TRY(hipMemcpyAsync(s->trace, s->h, hslice * 4, hipMemcpyDeviceToDevice, st));
    for (int l = 0; l < L; ++l) {
      const f3c_model::Block& bw = m->blk[l];
      const float* md = mod + (size_t)l * 6 * d;
      {
        Scope sc(s, F3C_PROF_LN, st, 0, lnb);
        HIP_TRY(launch_ln_mod(dt, s->h, rows, d, md, md + d, s->u, st));
      }
      {
        Scope sc(s, F3C_PROF_GEMM_QKV, st, 2.0 * rows * 3 * d * d, proj_bytes(3 * dd, dd, false));
        // queries stored times the attention's base-2 softmax scale (one rounding)
        HIP_TRY(launch_gemm(SITE_QKV, dt, EPI_STORE, rows, 3 * d, d, s->u, d, m->w(bw.qkv_w), d, m->b(bw.qkv_b),
                            nullptr, s->qkv, 3 * d, nullptr, 0, st, attention_q_scale(m->hd), d));
      }
      {
        double fl = 0;
        for (int g = 0; g < P * B; ++g)
          fl += 4.0 * (double)(tact.off[g + 1] - tact.off[g]) * (tact.off[g + 1] - tact.off[g]) * d;
        Scope sc(s, F3C_PROF_ATTN_SELF, st, fl, 4.0 * r * dd * E);
        const char* q = static_cast<const char*>(s->qkv);
        HIP_TRY(launch_attention(SITE_SELF, dt, m->cfg.heads, m->hd, tact, tact, q, 3 * d, q + d * es, 3 * d,
                                 q + 2 * d * es, 3 * d, s->att, d, s->ws, s->ws_bytes, st, true));
      }
      {
        Scope sc(s, F3C_PROF_GEMM_O, st, 2.0 * rows * d * d, proj_bytes(dd, dd, true));
        HIP_TRY(launch_gemm(SITE_O, dt, EPI_RESID, rows, d, d, s->att, d, m->w(bw.o_w), d, m->b(bw.o_b), md + 2 * d,
                            nullptr, 0, s->h, d, st));
      }
      if (s->sub_trace) {   // the same projection into a zeroed slice, without the gate
        float* sl = s->sub_trace + (size_t)(3 * l) * hslice;
        HIP_TRY(launch_zero(sl, hslice * 4, st));
        HIP_TRY(launch_gemm(SITE_OP, dt, EPI_RESID, rows, d, d, s->att, d, m->w(bw.o_w), d, m->b(bw.o_b), nullptr,
                            nullptr, 0, sl, d, st));
      }
      {
        Scope sc(s, F3C_PROF_LN, st, 0, lnb);
        HIP_TRY(launch_ln_mod(dt, s->h, rows, d, nullptr, nullptr, s->u, st));
      }
      {
        Scope sc(s, F3C_PROF_GEMM_Q, st, 2.0 * rows * d * d, proj_bytes(dd, dd, false));
        HIP_TRY(launch_gemm(SITE_Q, dt, EPI_STORE, rows, d, d, s->u, d, m->w(bw.q_w), d, m->b(bw.q_b), nullptr,
                            s->qc, d, nullptr, 0, st, attention_q_scale(m->hd), d));
      }
      {
        Scope sc(s, F3C_PROF_ATTN_CROSS, st, 4.0 * rows * m->Nc * d, (2.0 * r + 2.0 * cond_rows) * dd * E);
        const char* kv = static_cast<const char*>(s->kv) + (size_t)l * 2 * d * es;
        HIP_TRY(launch_attention(SITE_CROSS, dt, m->cfg.heads, m->hd, tact, cond_segs, s->qc, d, kv, 2 * L * d,
                                 kv + d * es, 2 * L * d, s->att, d, s->ws, s->ws_bytes, st, true));
      }
      {
        Scope sc(s, F3C_PROF_GEMM_CO, st, 2.0 * rows * d * d, proj_bytes(dd, dd, true));
        HIP_TRY(launch_gemm(SITE_CO, dt, EPI_RESID, rows, d, d, s->att, d, m->w(bw.co_w), d, m->b(bw.co_b), nullptr,
                            nullptr, 0, s->h, d, st));
      }
      if (s->sub_trace) {
        float* sl = s->sub_trace + (size_t)(3 * l + 1) * hslice;
        HIP_TRY(launch_zero(sl, hslice * 4, st));
        HIP_TRY(launch_gemm(SITE_OP, dt, EPI_RESID, rows, d, d, s->att, d, m->w(bw.co_w), d, m->b(bw.co_b), nullptr,
                            nullptr, 0, sl, d, st));
      }
      {
        Scope sc(s, F3C_PROF_LN, st, 0, lnb);
        HIP_TRY(launch_ln_mod(dt, s->h, rows, d, md + 3 * d, md + 4 * d, s->u, st));
      }
      {
        Scope sc(s, F3C_PROF_GEMM_FC1, st, 2.0 * rows * dm * d, proj_bytes(dm, dd, false));
        HIP_TRY(launch_gemm(SITE_FC1, dt, EPI_GELU, rows, dm, d, s->u, d, m->w(bw.fc1_w), d, m->b(bw.fc1_b), nullptr,
                            s->hid, dm, nullptr, 0, st));
      }
      {
        Scope sc(s, F3C_PROF_GEMM_FC2, st, 2.0 * rows * d * dm, proj_bytes(dd, dm, true));
        HIP_TRY(launch_gemm(SITE_FC2, dt, EPI_RESID, rows, d, dm, s->hid, dm, m->w(bw.fc2_w), dm, m->b(bw.fc2_b),
                            md + 5 * d, nullptr, 0, s->h, d, st));
      }
      if (s->sub_trace) {
        float* sl = s->sub_trace + (size_t)(3 * l + 2) * hslice;
        HIP_TRY(launch_zero(sl, hslice * 4, st));
        HIP_TRY(launch_gemm(SITE_OP, dt, EPI_RESID, rows, d, dm, s->hid, dm, m->w(bw.fc2_w), dm, m->b(bw.fc2_b), nullptr,
                            nullptr, 0, sl, d, st));
      }
      if (s->trace)
        HIP_TRY(hipMemcpyAsync(s->trace + (l + 1) * hslice, s->h, hslice * 4, hipMemcpyDeviceToDevice, st));
    }
    {
      Scope sc(s, F3C_PROF_FINAL, st, 0, rows * (d * 4.0 + 32));
      HIP_TRY(launch_final(dt, s->h, rows, d, m->w(m->top.out_w), m->b(m->top.out_b), s->vact, st));
    }
  }
  {
    Scope sc(s, F3C_PROF_EULER, st, 0, (double)B * N * 128 + P * arows * 32.0);
    const float dtf = (float)(t - t_next);
    const float ga = (float)(1.0 + w), gw = (float)w;
    HIP_TRY(launch_euler(x, v_cache, s->vact, guide ? s->vact + (size_t)arows * 8 : nullptr, ga, gw, pos, act, B, N,
                         dtf, v_prev, st));
  }
  s->cur = 1 - s->cur;
  s->last_act = act;
  s->last_mod = mod;
  s->last_selected = pos != nullptr;
  return F3C_OK;
}

}  // namespace

extern "C" {

const char* f3c_last_error(void) { return g_err.c_str(); }
int f3c_version(void) { return 1; }

int f3c_model_create(const f3c_model_cfg* cfg, f3c_model** out) {
  if (!out) return fail(F3C_EINVAL, "out is NULL");
  *out = nullptr;
  int rc = validate_cfg(cfg);
  if (rc) return rc;
  f3c_model* m = new f3c_model();
  m->cfg = *cfg;
  m->N = cfg->grid * cfg->grid * cfg->grid;
  m->d = cfg->width;
  m->hd = cfg->width / cfg->heads;
  m->dm = cfg->width * cfg->mlp_ratio;
  m->L = cfg->depth;
  m->dc = cfg->cond_width;
  m->Nc = cfg->cond_tokens;
  m->es = cfg->dtype == F3C_BF16 ? 2 : 4;
  const int d = m->d, dc = m->dc, dm = m->dm, L = m->L;
  auto add = [&](const std::string& n, int64_t r, int64_t c) { m->specs.push_back(Spec{n, r, c, c == 0}); };
  add("in_w", d, 8);
  add("in_b", d, 0);
  add("pos", m->N, d);
  add("t1_w", d, 256);
  add("t1_b", d, 0);
  add("t2_w", d, d);
  add("t2_b", d, 0);
  for (int l = 0; l < L; ++l) {
    const std::string p = "blk" + std::to_string(l) + ".";
    add(p + "mod_w", 6 * d, d);
    add(p + "mod_b", 6 * d, 0);
    add(p + "qkv_w", 3 * d, d);
    add(p + "qkv_b", 3 * d, 0);
    add(p + "o_w", d, d);
    add(p + "o_b", d, 0);
    add(p + "q_w", d, d);
    add(p + "q_b", d, 0);
    add(p + "kv_w", 2 * d, dc);
    add(p + "kv_b", 2 * d, 0);
    add(p + "co_w", d, d);
    add(p + "co_b", d, 0);
    add(p + "fc1_w", dm, d);
    add(p + "fc1_b", dm, 0);
    add(p + "fc2_w", d, dm);
    add(p + "fc2_b", d, 0);
  }
  add("out_w", 8, d);
  add("out_b", 8, 0);
  // Layout: per-block modulation and cross-attention K/V weights are grouped
  // across blocks so one GEMV / one GEMM serves all blocks.
  size_t off = 0;
  auto bytes_of = [&](const Spec& s) { return (size_t)s.numel() * (s.bias ? 4 : m->es); };
  m->mod_w = off;
  off = align256(off + (size_t)L * 6 * d * d * m->es);
  m->mod_b = off;
  off = align256(off + (size_t)L * 6 * d * 4);
  m->kv_w = off;
  off = align256(off + (size_t)L * 2 * d * dc * m->es);
  m->kv_b = off;
  off = align256(off + (size_t)L * 2 * d * 4);
  for (auto& s : m->specs) {
    const size_t dot = s.name.find('.');
    if (dot != std::string::npos) {
      const int l = std::stoi(s.name.substr(3, dot - 3));
      const std::string k = s.name.substr(dot + 1);
      if (k == "mod_w") { s.off = m->mod_w + (size_t)l * 6 * d * d * m->es; continue; }
      if (k == "mod_b") { s.off = m->mod_b + (size_t)l * 6 * d * 4; continue; }
      if (k == "kv_w") { s.off = m->kv_w + (size_t)l * 2 * d * dc * m->es; continue; }
      if (k == "kv_b") { s.off = m->kv_b + (size_t)l * 2 * d * 4; continue; }
    }
    s.off = off;
    off = align256(off + bytes_of(s));
  }
  m->wbytes = off;
  std::unordered_map<std::string, size_t> at;
  for (const auto& s : m->specs) at.emplace(s.name, s.off);
  m->top = {at.at("in_w"), at.at("in_b"), at.at("pos"), at.at("t1_w"), at.at("t1_b"),
            at.at("t2_w"), at.at("t2_b"), at.at("out_w"), at.at("out_b")};
  for (int l = 0; l < L; ++l) {
    const std::string p = "blk" + std::to_string(l) + ".";
    m->blk.push_back({at.at(p + "qkv_w"), at.at(p + "qkv_b"), at.at(p + "o_w"), at.at(p + "o_b"), at.at(p + "q_w"),
                      at.at(p + "q_b"), at.at(p + "co_w"), at.at(p + "co_b"), at.at(p + "fc1_w"), at.at(p + "fc1_b"),
                      at.at(p + "fc2_w"), at.at(p + "fc2_b")});
  }
  *out = m;
  return F3C_OK;
}

void f3c_model_destroy(f3c_model* m) { delete m; }

int f3c_weight_count(const f3c_model* m, int32_t* n) {
  if (!m || !n) return fail(F3C_EINVAL, "NULL argument");
  *n = (int32_t)m->specs.size();
  return F3C_OK;
}

int f3c_weight_info(const f3c_model* m, int32_t i, const char** name, int64_t* numel) {
  if (!m || !name || !numel) return fail(F3C_EINVAL, "NULL argument");
  if (i < 0 || i >= (int32_t)m->specs.size()) return fail(F3C_EINVAL, "weight index %d out of range", i);
  *name = m->specs[i].name.c_str();
  *numel = m->specs[i].numel();
  return F3C_OK;
}

int f3c_model_weights_bytes(const f3c_model* m, size_t* bytes) {
  if (!m || !bytes) return fail(F3C_EINVAL, "NULL argument");
  *bytes = m->wbytes;
  return F3C_OK;
}

int f3c_model_load_weights(f3c_model* m, void* weights_dev, size_t bytes, const float* const* host_f32, int32_t n) {
  if (!m || !weights_dev || !host_f32) return fail(F3C_EINVAL, "NULL argument");
  if ((uintptr_t)weights_dev & 255) return fail(F3C_EINVAL, "weights buffer must be 256-byte aligned");
  if (bytes < m->wbytes) return fail(F3C_ENOMEM, "weights buffer %zu < %zu bytes", bytes, m->wbytes);
  if (n != (int32_t)m->specs.size()) return fail(F3C_EINVAL, "expected %zu weight arrays, got %d", m->specs.size(), n);
  for (int32_t i = 0; i < n; ++i)
    if (!host_f32[i]) return fail(F3C_EINVAL, "weight %s is NULL", m->specs[i].name.c_str());
  std::vector<char> stage;
  char* dev = static_cast<char*>(weights_dev);
  // All blocks' modulation weights are stored input-major, [d][L*6d], for the
  // streaming GEMV; the other matrices keep their [out][in] layout.
  const int64_t d = m->d, R = (int64_t)m->L * 6 * d;
  std::vector<char> modt((size_t)(R * d) * m->es);
  for (int32_t i = 0; i < n; ++i) {
    const Spec& s = m->specs[i];
    const int64_t ne = s.numel();
    const size_t dot = s.name.find('.');
    if (dot != std::string::npos && s.name.substr(dot + 1) == "mod_w") {
      const int64_t l = std::stoll(s.name.substr(3, dot - 3));
      for (int64_t r = 0; r < 6 * d; ++r)
        for (int64_t k = 0; k < d; ++k) {
          const float v = host_f32[i][r * d + k];
          const size_t o = (size_t)(k * R + l * 6 * d + r);
          if (m->es == 2)
            reinterpret_cast<uint16_t*>(modt.data())[o] = f32_to_bf16_bits(v);
          else
            reinterpret_cast<float*>(modt.data())[o] = v;
        }
      continue;
    }
    if (s.bias || m->es == 4) {
      HIP_TRY(hipMemcpy(dev + s.off, host_f32[i], (size_t)ne * 4, hipMemcpyHostToDevice));
    } else {
      stage.resize((size_t)ne * 2);
      uint16_t* o = reinterpret_cast<uint16_t*>(stage.data());
      for (int64_t j = 0; j < ne; ++j) o[j] = f32_to_bf16_bits(host_f32[i][j]);
      HIP_TRY(hipMemcpy(dev + s.off, stage.data(), (size_t)ne * 2, hipMemcpyHostToDevice));
    }
  }
  HIP_TRY(hipMemcpy(dev + m->mod_w, modt.data(), modt.size(), hipMemcpyHostToDevice));
  m->wdev = dev;
  m->loaded = true;
  return F3C_OK;
}

double f3c_forward_flops(const f3c_model_cfg* c, int32_t n_tok, int32_t batch) {
  if (!c) return 0.0;
  return c->depth * block_flops(batch, n_tok, c->width, c->heads, c->cond_tokens, c->cond_width,
                                (double)c->width * c->mlp_ratio);
}

int f3c_state_bytes_ex(const f3c_model* m, int32_t batch, uint32_t flags, size_t* bytes) {
  if (!m || !bytes) return fail(F3C_EINVAL, "NULL argument");
  if (flags & ~(uint32_t)F3C_STATE_GUIDED) return fail(F3C_EINVAL, "unknown state flags 0x%x", flags);
  const int P = (flags & F3C_STATE_GUIDED) ? 2 : 1;
  if (batch < 1 || batch * P > F3C_MAX_BATCH)
    return fail(F3C_EINVAL, "batch must be in 1..%d%s", F3C_MAX_BATCH / P, P == 2 ? " for a guided state" : "");
  const size_t R = (size_t)batch * m->N, A = P * R, d = m->d, es = m->es;
  size_t t = 0;
  t += 2 * align256(R * 32);                   // velocity cache pair
  t += align256(A * d * 4);                    // h
  t += 3 * align256(A * d * es);               // u, att, qc
  t += align256(A * 3 * d * es);               // qkv
  t += align256(A * m->dm * es);               // mlp hidden
  t += align256(A * 32);                       // v_act
  t += 3 * align256(R * 4);                    // idx, pos, score
  t += align256(select_workspace_bytes(batch, m->N));   // selection workspace
  t += align256((size_t)m->L * 6 * d * 4);     // mod
  t += align256(2 * d * 4);                    // temb scratch
  t += align256((size_t)P * batch * m->Nc * m->dc * es);            // condition tokens
  t += align256((size_t)P * batch * m->Nc * 2 * m->L * d * es);     // cross K/V, all blocks
  t += kAttnWsBytes;                                                  // attention split partials
  *bytes = t;
  return F3C_OK;
}

int f3c_state_bytes(const f3c_model* m, int32_t batch, size_t* bytes) { return f3c_state_bytes_ex(m, batch, 0, bytes); }

int f3c_state_create_ex(f3c_model* m, int32_t batch, uint32_t flags, void* state_dev, size_t bytes,
                        f3c_stream stream, f3c_state** out) {
  if (!m || !state_dev || !out) return fail(F3C_EINVAL, "NULL argument");
  *out = nullptr;
  size_t need = 0;
  int rc = f3c_state_bytes_ex(m, batch, flags, &need);
  if (rc) return rc;
  if ((uintptr_t)state_dev & 255) return fail(F3C_EINVAL, "state buffer must be 256-byte aligned");
  if (bytes < need) return fail(F3C_ENOMEM, "state buffer %zu < %zu bytes", bytes, need);
  f3c_state* s = new f3c_state();
  s->m = m;
  s->B = batch;
  s->guided = (flags & F3C_STATE_GUIDED) != 0;
  s->dev = static_cast<char*>(state_dev);
  s->bytes = bytes;
  const size_t P = s->guided ? 2 : 1;
  const size_t R = (size_t)batch * m->N, A = P * R, d = m->d, es = m->es;
  char* p = s->dev;
  auto take = [&](size_t n) { char* r = p; p += align256(n); return r; };
  s->v[0] = (float*)take(R * 32);
  s->v[1] = (float*)take(R * 32);
  s->h = (float*)take(A * d * 4);
  s->u = take(A * d * es);
  s->att = take(A * d * es);
  s->qc = take(A * d * es);
  s->qkv = take(A * 3 * d * es);
  s->hid = take(A * m->dm * es);
  s->vact = (float*)take(A * 32);
  s->idx = (int32_t*)take(R * 4);
  s->pos = (int32_t*)take(R * 4);
  s->score = (float*)take(R * 4);
  s->sel_ws = take(select_workspace_bytes(batch, m->N));
  s->mod = (float*)take((size_t)m->L * 6 * d * 4);
  s->temb = (float*)take(2 * d * 4);
  s->cond_t = take(P * batch * m->Nc * m->dc * es);
  s->kv = take(P * batch * m->Nc * 2 * m->L * d * es);
  s->ws = (float*)take(kAttnWsBytes);
  s->ws_bytes = kAttnWsBytes;
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = f3c::launch_zero(s->v[0], R * 32, st);
  if (e == hipSuccess) e = f3c::launch_zero(s->v[1], R * 32, st);
  if (e != hipSuccess) {
    delete s;
    return fail(F3C_EHIP, "zeroing caches: %s", hipGetErrorString(e));
  }
  *out = s;
  return F3C_OK;
}

int f3c_state_create(f3c_model* m, int32_t batch, void* state_dev, size_t bytes, f3c_stream stream,
                     f3c_state** out) {
  return f3c_state_create_ex(m, batch, 0, state_dev, bytes, stream, out);
}

void f3c_state_destroy(f3c_state* s) {
  if (!s) return;
  for (auto& p : s->prof)
    for (auto e : p.ev) (void)hipEventDestroy(e);
  for (auto e : s->pool) (void)hipEventDestroy(e);
  delete s;
}

int f3c_state_reset(f3c_state* s, f3c_stream stream) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  const size_t R = (size_t)s->B * s->m->N;
  HIP_TRY(f3c::launch_zero(s->v[0], R * 32, (hipStream_t)stream));
  HIP_TRY(f3c::launch_zero(s->v[1], R * 32, (hipStream_t)stream));
  s->cur = 0;
  return F3C_OK;
}

int f3c_state_set_omega(f3c_state* s, float omega) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (!(omega >= 0.0f && omega <= 1.0f)) return fail(F3C_EINVAL, "omega must be in [0, 1]");
  s->omega = omega;
  return F3C_OK;
}

namespace {

// Condition tokens of one pass ([B][Nc][dc] f32) -> the cross-attention K/V of
// every block, stored at rows half * B * Nc of the state's K/V buffer.
int cond_kv(f3c_state* s, const float* cond_dev, int half, hipStream_t st) {
  f3c_model* m = s->m;
  const int rows = s->B * m->Nc, n = 2 * m->L * m->d;
  char* ct = static_cast<char*>(s->cond_t) + (size_t)half * rows * m->dc * m->es;
  char* kv = static_cast<char*>(s->kv) + (size_t)half * rows * n * m->es;
  Scope sc(s, F3C_PROF_COND, st, 2.0 * rows * n * m->dc, 0);
  HIP_TRY(launch_convert(m->cfg.dtype, cond_dev, ct, (int64_t)rows * m->dc, st));
  HIP_TRY(launch_gemm(SITE_COND, m->cfg.dtype, EPI_STORE, rows, n, m->dc, ct, m->dc, m->wdev + m->kv_w, m->dc,
                      (const float*)(m->wdev + m->kv_b), nullptr, kv, n, nullptr, 0, st));
  return F3C_OK;
}

}  // namespace

int f3c_set_cond(f3c_state* s, const float* cond_dev, f3c_stream stream) {
  int rc = check_state(s);
  if (rc) return rc;
  if (!cond_dev) return fail(F3C_EINVAL, "cond is NULL");
  if ((rc = cond_kv(s, cond_dev, 0, (hipStream_t)stream))) return rc;
  s->cond_set = true;
  return F3C_OK;
}

int f3c_set_uncond(f3c_state* s, const float* uncond_dev, f3c_stream stream) {
  int rc = check_state(s);
  if (rc) return rc;
  if (!s->guided) return fail(F3C_ESTATE, "state was not created with F3C_STATE_GUIDED");
  if (!uncond_dev) return fail(F3C_EINVAL, "uncond is NULL");
  if ((rc = cond_kv(s, uncond_dev, 1, (hipStream_t)stream))) return rc;
  s->uncond_set = true;
  return F3C_OK;
}

int f3c_plan_bytes(const f3c_model* m, int32_t n, size_t* bytes) {
  if (!m || !bytes) return fail(F3C_EINVAL, "NULL argument");
  if (n < 0 || n > F3C_MAX_PLAN) return fail(F3C_EINVAL, "plan of %d times outside 0..%d", n, F3C_MAX_PLAN);
  *bytes = align256((size_t)n * 6 * m->L * m->d * 4) + align256((size_t)n * 2 * m->d * 4);
  return F3C_OK;
}

int f3c_state_plan_times(f3c_state* s, const double* t_host, int32_t n, void* plan_dev, size_t bytes,
                         f3c_stream stream) {
  int rc = check_state(s);
  if (rc) return rc;
  size_t need = 0;
  if ((rc = f3c_plan_bytes(s->m, n, &need))) return rc;
  if (n == 0) {
    s->plan_t.clear();
    s->plan_mod = nullptr;
    return F3C_OK;
  }
  if (!t_host || !plan_dev) return fail(F3C_EINVAL, "NULL argument");
  for (int32_t i = 0; i < n; ++i)
    if (!std::isfinite(t_host[i])) return fail(F3C_EINVAL, "plan time %d is not finite", i);
  if ((uintptr_t)plan_dev & 255) return fail(F3C_EINVAL, "plan buffer must be 256-byte aligned");
  if (bytes < need) return fail(F3C_ENOMEM, "plan buffer %zu < %zu bytes", bytes, need);
  f3c_model* m = s->m;
  const int d = m->d, L = m->L, dt = m->cfg.dtype, R = 6 * L * d;
  const size_t es = m->es;
  float* mod = static_cast<float*>(plan_dev);
  float* temb = reinterpret_cast<float*>(static_cast<char*>(plan_dev) + align256((size_t)n * R * 4));
  hipStream_t st = (hipStream_t)stream;
  s->plan_t.clear();                     // no step may read a half-enqueued plan
  s->plan_mod = nullptr;
  {
    const int passes = (n + 7) / 8;
    Scope sc(s, F3C_PROF_MOD, st, 0, (double)es * d * ((256.0 + d) * n + (double)R * passes));
    const char* mw = m->wdev;
    for (int32_t i = 0; i < n; ++i) {
      float* e = temb + (size_t)i * 2 * d;
      HIP_TRY(launch_gemv(dt, m->w(m->top.t1_w), m->b(m->top.t1_b), nullptr, t_host[i], GEMV_IN_TIMESTEP, 1, d, 256, e,
                          st));
      HIP_TRY(launch_gemv(dt, m->w(m->top.t2_w), m->b(m->top.t2_b), e, 0.0, GEMV_IN_PLAIN, 0, d, d, e + d, st));
    }
    for (int32_t c = 0; c < n; c += 8)
      HIP_TRY(launch_gemv_tn(dt, mw + m->mod_w, (const float*)(mw + m->mod_b), temb + (size_t)c * 2 * d + d, 2 * d,
                             std::min(8, n - c), R, d, mod + (size_t)c * R, R, st));
  }
  s->plan_t.assign(t_host, t_host + n);
  s->plan_mod = mod;
  return F3C_OK;
}

static int step_common(f3c_state* s, float* x, double t, double t_next, const int32_t* n_cache, bool guide, double w,
                       f3c_stream stream) {
  int rc = check_state(s);
  if (rc) return rc;
  if (!s->cond_set) return fail(F3C_ESTATE, "condition not set (call f3c_set_cond first)");
  if (!x) return fail(F3C_EINVAL, "x is NULL");
  if (!std::isfinite(t) || !std::isfinite(t_next) || !(t > t_next))
    return fail(F3C_EINVAL, "need finite t > t_next (got %g, %g)", t, t_next);
  if (n_cache)
    for (int b = 0; b < s->B; ++b)
      if (n_cache[b] < 0 || n_cache[b] > s->m->N)
        return fail(F3C_EINVAL, "n_cache[%d] = %d outside [0, %d]", b, n_cache[b], s->m->N);
  if (s->trace || s->sub_trace) {
    size_t rows = 0;
    for (int b = 0; b < s->B; ++b) rows += s->m->N - (n_cache ? n_cache[b] : 0);
    const size_t slice = rows * (guide ? 2 : 1) * s->m->d * sizeof(float);
    if (s->trace && (size_t)(s->m->L + 1) * slice > s->trace_bytes)
      return fail(F3C_ENOMEM, "trace buffer %zu < %zu bytes", s->trace_bytes, (size_t)(s->m->L + 1) * slice);
    if (s->sub_trace && (size_t)(3 * s->m->L) * slice > s->sub_trace_bytes)
      return fail(F3C_ENOMEM, "sublayer trace buffer %zu < %zu bytes", s->sub_trace_bytes,
                  (size_t)(3 * s->m->L) * slice);
  }
  if (guide) {
    if (!s->guided) return fail(F3C_ESTATE, "state was not created with F3C_STATE_GUIDED");
    if (!s->uncond_set) return fail(F3C_ESTATE, "unconditional input not set (call f3c_set_uncond first)");
    if (!std::isfinite(w)) return fail(F3C_EINVAL, "guidance weight must be finite");
  }
  return run_step(s, x, t, t_next, n_cache, guide, w, (hipStream_t)stream);
}

int f3c_full_step(f3c_state* s, float* x_dev, double t, double t_next, f3c_stream stream) {
  return step_common(s, x_dev, t, t_next, nullptr, false, 0.0, stream);
}

int f3c_cached_step(f3c_state* s, float* x_dev, double t, double t_next, const int32_t* n_cache_host,
                    f3c_stream stream) {
  if (!n_cache_host) return fail(F3C_EINVAL, "n_cache is NULL");
  return step_common(s, x_dev, t, t_next, n_cache_host, false, 0.0, stream);
}

int f3c_guided_step(f3c_state* s, float* x_dev, double t, double t_next, const int32_t* n_cache_host, double w,
                    f3c_stream stream) {
  return step_common(s, x_dev, t, t_next, n_cache_host, true, w, stream);
}

int f3c_state_views(const f3c_state* s, float** v_cache, float** v_prev, int32_t** idx_active, int32_t** pos,
                    float** v_act, float** mod, float** score, int32_t* act_off_host) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (v_cache) *v_cache = s->v[s->cur];
  if (v_prev) *v_prev = s->v[1 - s->cur];
  if (idx_active) *idx_active = s->last_selected ? s->idx : nullptr;
  if (pos) *pos = s->last_selected ? s->pos : nullptr;
  if (v_act) *v_act = s->vact;
  if (mod) *mod = const_cast<float*>(s->last_mod ? s->last_mod : s->mod);
  if (score) *score = s->score;
  if (act_off_host)
    for (int b = 0; b <= s->B; ++b) act_off_host[b] = s->last_act.off[b];
  return F3C_OK;
}

int f3c_state_trace_blocks(f3c_state* s, float* h_trace_dev, size_t bytes) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (h_trace_dev && ((uintptr_t)h_trace_dev & 15)) return fail(F3C_EINVAL, "trace buffer must be 16-byte aligned");
  s->trace = h_trace_dev;
  s->trace_bytes = h_trace_dev ? bytes : 0;
  return F3C_OK;
}

int f3c_state_trace_sublayers(f3c_state* s, float* trace_dev, size_t bytes) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (trace_dev && ((uintptr_t)trace_dev & 15)) return fail(F3C_EINVAL, "trace buffer must be 16-byte aligned");
  s->sub_trace = trace_dev;
  s->sub_trace_bytes = trace_dev ? bytes : 0;
  return F3C_OK;
}

int f3c_debug_force_active(f3c_state* s, const int32_t* idx_active_dev) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (idx_active_dev && ((uintptr_t)idx_active_dev & 3)) return fail(F3C_EINVAL, "index buffer must be 4-byte aligned");
  s->force_idx = idx_active_dev;
  return F3C_OK;
}

int f3c_state_record_scores(f3c_state* s, int32_t on) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  s->record_scores = on != 0;
  return F3C_OK;
}

int f3c_state_export(const f3c_state* s, float* host, size_t n_floats, f3c_stream stream) {
  if (!s || !host) return fail(F3C_EINVAL, "NULL argument");
  const size_t R = (size_t)s->B * s->m->N * 8;
  if (n_floats < 2 * R) return fail(F3C_ENOMEM, "host buffer holds %zu < %zu floats", n_floats, 2 * R);
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(hipMemcpyAsync(host, s->v[s->cur], R * 4, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipMemcpyAsync(host + R, s->v[1 - s->cur], R * 4, hipMemcpyDeviceToHost, st));
  HIP_TRY(hipStreamSynchronize(st));
  return F3C_OK;
}

int f3c_state_import(f3c_state* s, const float* host, size_t n_floats, f3c_stream stream) {
  if (!s || !host) return fail(F3C_EINVAL, "NULL argument");
  const size_t R = (size_t)s->B * s->m->N * 8;
  if (n_floats < 2 * R) return fail(F3C_ENOMEM, "host buffer holds %zu < %zu floats", n_floats, 2 * R);
  hipStream_t st = (hipStream_t)stream;
  HIP_TRY(hipMemcpyAsync(s->v[s->cur], host, R * 4, hipMemcpyHostToDevice, st));
  HIP_TRY(hipMemcpyAsync(s->v[1 - s->cur], host + R, R * 4, hipMemcpyHostToDevice, st));
  HIP_TRY(hipStreamSynchronize(st));
  return F3C_OK;
}

int f3c_profile_enable(f3c_state* s, uint32_t mask) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  s->prof_mask = mask & ((1u << F3C_PROF_CLASSES) - 1u);
  return F3C_OK;
}

int f3c_profile_read(f3c_state* s, int32_t cls, int64_t* launches, double* ms, double* flops, double* bytes) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  if (cls < 0 || cls >= F3C_PROF_CLASSES) return fail(F3C_EINVAL, "class %d out of range", cls);
  Prof& p = s->prof[cls];
  double total = 0;
  for (size_t i = 0; i + 1 < p.ev.size(); i += 2) {
    HIP_TRY(hipEventSynchronize(p.ev[i + 1]));
    float t = 0;
    HIP_TRY(hipEventElapsedTime(&t, p.ev[i], p.ev[i + 1]));
    total += t;
  }
  if (launches) *launches = p.launches;
  if (ms) *ms = total;
  if (flops) *flops = p.flops;
  if (bytes) *bytes = p.bytes;
  return F3C_OK;
}

int f3c_profile_reset(f3c_state* s) {
  if (!s) return fail(F3C_EINVAL, "state is NULL");
  for (auto& p : s->prof) {
    for (auto e : p.ev) {
      (void)hipEventSynchronize(e);
      s->pool.push_back(e);
    }
    p.ev.clear();
    p.launches = 0;
    p.flops = p.bytes = 0;
  }
  return F3C_OK;
}

// ------------------------------------------------------------ operator entries

int f3c_op_select_workspace_bytes(int32_t batch, int32_t n_tokens, size_t* bytes) {
  if (!bytes) return fail(F3C_EINVAL, "NULL argument");
  if (batch < 1 || batch > F3C_MAX_BATCH) return fail(F3C_EINVAL, "batch must be in 1..%d", F3C_MAX_BATCH);
  if (n_tokens < 1 || n_tokens > F3C_MAX_TOKENS) return fail(F3C_EINVAL, "n_tokens must be in 1..%d", F3C_MAX_TOKENS);
  *bytes = select_workspace_bytes(batch, n_tokens);
  return F3C_OK;
}

namespace {

int select_args(int32_t batch, int32_t n_tokens, const float* v_cache, const float* v_prev, float omega,
                const int32_t* n_cache_host, int32_t* idx_active, int32_t* pos, Segs* quota, Segs* act) {
  if (batch < 1 || batch > F3C_MAX_BATCH) return fail(F3C_EINVAL, "batch must be in 1..%d", F3C_MAX_BATCH);
  if (n_tokens < 1 || n_tokens > F3C_MAX_TOKENS) return fail(F3C_EINVAL, "n_tokens must be in 1..%d", F3C_MAX_TOKENS);
  if (!v_cache || !v_prev || !n_cache_host || !idx_active || !pos) return fail(F3C_EINVAL, "NULL argument");
  if (!(omega >= 0.0f && omega <= 1.0f)) return fail(F3C_EINVAL, "omega must be in [0, 1]");
  *quota = Segs{};
  *act = Segs{};
  quota->B = act->B = batch;
  for (int b = 0; b < batch; ++b) {
    const int c = n_cache_host[b];
    if (c < 0 || c > n_tokens) return fail(F3C_EINVAL, "n_cache[%d] = %d outside [0, %d]", b, c, n_tokens);
    quota->off[b] = c;
    act->off[b + 1] = act->off[b] + n_tokens - c;
  }
  return F3C_OK;
}

}  // namespace

int f3c_op_select(int32_t batch, int32_t n_tokens, const float* v_cache, const float* v_prev, float omega,
                  const int32_t* n_cache_host, int32_t* idx_active, int32_t* pos, float* score, void* workspace,
                  size_t workspace_bytes, f3c_stream stream) {
  Segs quota, act;
  if (int rc = select_args(batch, n_tokens, v_cache, v_prev, omega, n_cache_host, idx_active, pos, &quota, &act))
    return rc;
  if (!workspace || ((uintptr_t)workspace & 255)) return fail(F3C_EINVAL, "workspace must be a 256-byte aligned buffer");
  const size_t need = select_workspace_bytes(batch, n_tokens);
  if (workspace_bytes < need) return fail(F3C_ENOMEM, "workspace %zu < %zu bytes", workspace_bytes, need);
  HIP_TRY(launch_select(v_cache, v_prev, batch, n_tokens, omega, 1.0f - omega, quota, act, idx_active, pos, score,
                        workspace, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_select_scores(int32_t batch, int32_t n_tokens, const float* scores, const int32_t* n_cache_host,
                         int32_t* idx_active, int32_t* pos, f3c_stream stream) {
  Segs quota, act;
  // the same shape and quota checks as f3c_op_select, with the scores in place of the two caches
  if (int rc = select_args(batch, n_tokens, scores, scores, 0.0f, n_cache_host, idx_active, pos, &quota, &act))
    return rc;
  HIP_TRY(launch_select_scores(scores, batch, n_tokens, quota, act, idx_active, pos, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_select_noalloc(int32_t batch, int32_t n_tokens, const float* v_cache, const float* v_prev, float omega,
                          const int32_t* n_cache_host, int32_t* idx_active, int32_t* pos, float* score,
                          f3c_stream stream) {
  Segs quota, act;
  if (int rc = select_args(batch, n_tokens, v_cache, v_prev, omega, n_cache_host, idx_active, pos, &quota, &act))
    return rc;
  if ((int64_t)batch * n_tokens > F3C_NOALLOC_MAX_TOKENS)
    return fail(F3C_EINVAL, "batch %d x %d tokens exceeds the static scratch's %d tokens", batch, n_tokens,
                F3C_NOALLOC_MAX_TOKENS);
  void* scratch = nullptr;
  size_t have = 0;
  HIP_TRY(select_static_scratch(&scratch, &have));
  const size_t need = select_workspace_bytes(batch, n_tokens);
  if (need > have) return fail(F3C_EINVAL, "selection scratch %zu > static %zu bytes", need, have);
  HIP_TRY(launch_select(v_cache, v_prev, batch, n_tokens, omega, 1.0f - omega, quota, act, idx_active, pos, score,
                        scratch, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_gemm(int32_t dtype, int32_t epilogue, int32_t M, int32_t N, int32_t K, const void* A, int32_t lda,
                const void* W, int32_t ldw, const float* bias, const float* gate, void* out, int32_t ldo,
                float* resid, int32_t ldr, f3c_stream stream) {
  if (dtype != F3C_F32 && dtype != F3C_BF16) return fail(F3C_EINVAL, "bad dtype");
  if (epilogue < 0 || epilogue > 2) return fail(F3C_EINVAL, "bad epilogue");
  const int es = dtype == F3C_BF16 ? 2 : 4;
  if (M < 0 || N <= 0 || K <= 0) return fail(F3C_EINVAL, "bad shape");
  if (N % 128) return fail(F3C_EINVAL, "N must be a multiple of 128");
  if ((K * es) % 128) return fail(F3C_EINVAL, "K must be a multiple of %d", 128 / es);
  if (lda < K || ldw < K || (lda * es) % 16 || (ldw * es) % 16) return fail(F3C_EINVAL, "bad leading dims");
  if (!A || !W || !bias) return fail(F3C_EINVAL, "NULL operand");
  if (epilogue == 2 ? (!resid || ldr < N || ldr % 4) : (!out || ldo < N || ldo % 4))
    return fail(F3C_EINVAL, "bad output (leading dim below N or not a multiple of 4)");
  HIP_TRY(launch_gemm(SITE_OP, dtype, epilogue, M, N, K, A, lda, W, ldw, bias, gate, out, ldo, resid, ldr,
                      (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_attention(int32_t dtype, int32_t heads, int32_t head_dim, int32_t batch, const int32_t* q_off_host,
                     const int32_t* k_off_host, const void* q, int32_t ldq, const void* k, int32_t ldk,
                     const void* v, int32_t ldv, void* o, int32_t ldo, float* workspace, size_t workspace_bytes,
                     int32_t q_prescaled, f3c_stream stream) {
  if (dtype != F3C_F32 && dtype != F3C_BF16) return fail(F3C_EINVAL, "bad dtype");
  if (head_dim != 32 && head_dim != 64) return fail(F3C_EINVAL, "head_dim must be 32 or 64");
  if (q_prescaled != 0 && q_prescaled != 1) return fail(F3C_EINVAL, "q_prescaled must be 0 or 1");
  if (heads < 1 || heads > 65535) return fail(F3C_EINVAL, "bad heads");
  if (batch < 1 || batch > F3C_MAX_BATCH) return fail(F3C_EINVAL, "batch must be in 1..%d", F3C_MAX_BATCH);
  if (!q_off_host || !k_off_host || !q || !k || !v || !o) return fail(F3C_EINVAL, "NULL argument");
  const int es = dtype == F3C_BF16 ? 2 : 4, w = heads * head_dim;
  if (ldq < w || ldk < w || ldv < w || ldo < w) return fail(F3C_EINVAL, "leading dims below heads*head_dim");
  if ((ldq * es) % 16 || (ldk * es) % 16 || (ldv * es) % 16) return fail(F3C_EINVAL, "rows must be 16-byte aligned");
  Segs qs{}, ks{};
  qs.B = ks.B = batch;
  for (int b = 0; b <= batch; ++b) {
    qs.off[b] = q_off_host[b];
    ks.off[b] = k_off_host[b];
    if (b > 0 && (qs.off[b] < qs.off[b - 1] || ks.off[b] < ks.off[b - 1]))
      return fail(F3C_EINVAL, "offsets must be non-decreasing");
  }
  if (qs.off[0] < 0 || ks.off[0] < 0) return fail(F3C_EINVAL, "negative offset");
  for (int b = 0; b < batch; ++b)
    if (qs.off[b + 1] > qs.off[b] && ks.off[b + 1] == ks.off[b])
      return fail(F3C_EINVAL, "sample %d has queries but no keys", b);
  if (workspace && ((uintptr_t)workspace & 15)) return fail(F3C_EINVAL, "workspace must be 16-byte aligned");
  if (dtype == F3C_BF16 && head_dim == 64) {
    // the bf16 64-wide kernel addresses one sample's key and value rows with 32-bit offsets
    int64_t nk_max = 0;
    for (int b = 0; b < batch; ++b) nk_max = std::max<int64_t>(nk_max, ks.off[b + 1] - ks.off[b]);
    const int64_t span = ((nk_max + 63) / 64) * 64 * (int64_t)std::max(ldk, ldv) * 2;
    if (span >= (int64_t(1) << 31)) return fail(F3C_EINVAL, "one sample's key rows span 2 GiB or more");
  }
  HIP_TRY(launch_attention(SITE_OP, dtype, heads, head_dim, qs, ks, q, ldq, k, ldk, v, ldv, o, ldo, workspace,
                           workspace ? workspace_bytes : 0, (hipStream_t)stream, q_prescaled == 1));
  return F3C_OK;
}

int f3c_op_ln_mod(int32_t dtype, int32_t rows, int32_t d, const float* h, const float* shift, const float* scale,
                  void* out, f3c_stream stream) {
  if (dtype != F3C_F32 && dtype != F3C_BF16) return fail(F3C_EINVAL, "bad dtype");
  if (rows < 0 || !h || !out) return fail(F3C_EINVAL, "bad argument");
  if (d != 128 && d != 256 && d != 512 && d != 1024 && d != 2048) return fail(F3C_EINVAL, "unsupported d %d", d);
  if ((shift == nullptr) != (scale == nullptr)) return fail(F3C_EINVAL, "shift and scale go together");
  HIP_TRY(launch_ln_mod(dtype, h, rows, d, shift, scale, out, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_modulation(const f3c_model* m, double t, float* mod_dev, float* scratch_dev, f3c_stream stream) {
  if (!m || !mod_dev || !scratch_dev) return fail(F3C_EINVAL, "NULL argument");
  if (!m->loaded) return fail(F3C_ESTATE, "weights not loaded");
  if (!std::isfinite(t)) return fail(F3C_EINVAL, "t must be finite");
  hipStream_t st = (hipStream_t)stream;
  const int d = m->d, dt = m->cfg.dtype;
  HIP_TRY(launch_gemv(dt, m->w(m->top.t1_w), m->b(m->top.t1_b), nullptr, t, GEMV_IN_TIMESTEP, 1, d, 256, scratch_dev, st));
  HIP_TRY(launch_gemv(dt, m->w(m->top.t2_w), m->b(m->top.t2_b), scratch_dev, 0.0, GEMV_IN_PLAIN, 0, d, d, scratch_dev + d, st));
  HIP_TRY(launch_gemv_t(dt, m->wdev + m->mod_w, (const float*)(m->wdev + m->mod_b), scratch_dev + d, 6 * m->L * d, d,
                        mod_dev, st));
  return F3C_OK;
}

// Segment table from B+1 host offsets; each segment at most `cap` rows.
static int segs_from_host(int32_t batch, const int32_t* off_host, int cap, Segs* out) {
  if (batch < 1 || batch > F3C_MAX_BATCH) return fail(F3C_EINVAL, "batch must be in 1..%d", F3C_MAX_BATCH);
  if (!off_host) return fail(F3C_EINVAL, "NULL offsets");
  out->B = batch;
  for (int b = 0; b <= batch; ++b) {
    out->off[b] = off_host[b];
    if (b == 0 && off_host[0] < 0) return fail(F3C_EINVAL, "negative offset");
    if (b > 0 && (off_host[b] < off_host[b - 1] || off_host[b] - off_host[b - 1] > cap))
      return fail(F3C_EINVAL, "segment %d must hold 0..%d rows", b - 1, cap);
  }
  return F3C_OK;
}

int f3c_op_embed(const f3c_model* m, int32_t batch, const float* x, const int32_t* idx_active,
                 const int32_t* act_off_host, float* h, f3c_stream stream) {
  if (!m || !x || !h) return fail(F3C_EINVAL, "NULL argument");
  if (!m->loaded) return fail(F3C_ESTATE, "weights not loaded");
  Segs act{};
  if (int rc = segs_from_host(batch, act_off_host, m->N, &act)) return rc;
  if (act.off[0] != 0) return fail(F3C_EINVAL, "act_off[0] must be 0");
  if (!idx_active)
    for (int b = 0; b < batch; ++b)
      if (act.off[b + 1] - act.off[b] != m->N) return fail(F3C_EINVAL, "without idx_active every token is active");
  HIP_TRY(launch_embed(m->cfg.dtype, x, m->N, idx_active, act, m->w(m->top.in_w), m->b(m->top.in_b), m->w(m->top.pos), m->d, h,
                       0, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_final(const f3c_model* m, int32_t rows, const float* h, float* v_act, f3c_stream stream) {
  if (!m || !h || !v_act || rows < 0) return fail(F3C_EINVAL, "bad argument");
  if (!m->loaded) return fail(F3C_ESTATE, "weights not loaded");
  HIP_TRY(launch_final(m->cfg.dtype, h, rows, m->d, m->w(m->top.out_w), m->b(m->top.out_b), v_act, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_euler(int32_t batch, int32_t n_tokens, float* x, const float* v_cache, const float* v_act,
                 const int32_t* pos, const int32_t* act_off_host, double t, double t_next, float* v_new,
                 f3c_stream stream) {
  if (!x || !v_cache || !v_new) return fail(F3C_EINVAL, "NULL argument");
  if (n_tokens < 1) return fail(F3C_EINVAL, "n_tokens must be positive");
  if (v_new == v_cache) return fail(F3C_EINVAL, "v_new must not alias v_cache");
  if (!std::isfinite(t) || !std::isfinite(t_next)) return fail(F3C_EINVAL, "t and t_next must be finite");
  Segs act{};
  if (int rc = segs_from_host(batch, act_off_host, n_tokens, &act)) return rc;
  if (act.off[batch] > act.off[0] && !v_act) return fail(F3C_EINVAL, "active rows need v_act");
  if (!pos)
    for (int b = 0; b < batch; ++b)
      if (act.off[b + 1] - act.off[b] != n_tokens) return fail(F3C_EINVAL, "without pos every token is active");
  const float dtf = (float)(t - t_next);
  HIP_TRY(launch_euler(x, v_cache, v_act, nullptr, 0.0f, 0.0f, pos, act, batch, n_tokens, dtf, v_new,
                       (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_pack_occupancy(int32_t batch, int64_t n_voxels, const float* logits, uint32_t* bits, f3c_stream stream) {
  if (!logits || !bits) return fail(F3C_EINVAL, "NULL argument");
  if (batch < 1 || batch > 65535) return fail(F3C_EINVAL, "batch must be in 1..65535");
  if (n_voxels < 1 || n_voxels > (int64_t(1) << 36)) return fail(F3C_EINVAL, "n_voxels must be in 1..2^36");
  HIP_TRY(launch_pack_occupancy(logits, batch, n_voxels, bits, (hipStream_t)stream));
  return F3C_OK;
}

int f3c_op_dynamic_voxels(int32_t batch, int64_t n_words, const uint32_t* occ_next, const uint32_t* occ_prev,
                          int64_t* counts, f3c_stream stream) {
  if (!occ_next || !occ_prev || !counts) return fail(F3C_EINVAL, "NULL argument");
  if (batch < 1 || batch > 65535) return fail(F3C_EINVAL, "batch must be in 1..65535");
  if (n_words < 1) return fail(F3C_EINVAL, "n_words must be positive");
  HIP_TRY(launch_dynamic_voxels(occ_next, occ_prev, batch, n_words, counts, (hipStream_t)stream));
  return F3C_OK;
}

// ------------------------------------------------------------ host schedules

static double shift_time(double u, double eta) { return eta * u / (1.0 + (eta - 1.0) * u); }

int f3c_time_grid(int32_t steps, double eta, double* out_host) {
  if (steps < 1 || !out_host) return fail(F3C_EINVAL, "need steps >= 1 and an output array");
  if (!(eta > 0.0) || !std::isfinite(eta)) return fail(F3C_EINVAL, "eta must be positive and finite");
  for (int k = 0; k <= steps; ++k) out_host[k] = shift_time(1.0 - (double)k / steps, eta);
  return F3C_OK;
}

int32_t f3c_guidance_active(double t, double lo, double hi) { return (lo <= t && t <= hi) ? 1 : 0; }

// The schedule's ratios (rho_a, rho_CFG-OFF, xi) are decimals in the paper
// (0.2, 0.75, 0.7). A double argument stands for the shortest decimal that
// rounds to it (0.2 means 1/5 exactly, 0.2000000001 means 2000000001/10^10),
// and the ceilings and floors of Algorithm 1 are taken exactly on that
// decimal, in integer arithmetic.
namespace {

struct Decimal {
  uint64_t mant;   // value = mant * 10^exp10
  int exp10;
};

// Digit string of `prec` significant digits -> (mantissa, exponent), from
// the "%.*e" form d.ddde[+-]xx of a positive finite value.
bool parse_sci(const char* buf, Decimal* out) {
  uint64_t m = 0;
  int digits_after_point = 0, seen_point = 0;
  const char* p = buf;
  for (; *p && *p != 'e'; ++p) {
    if (*p == '.') { seen_point = 1; continue; }
    if (*p < '0' || *p > '9') return false;
    m = m * 10 + (uint64_t)(*p - '0');
    digits_after_point += seen_point;
  }
  if (*p != 'e') return false;
  out->mant = m;
  out->exp10 = std::atoi(p + 1) - digits_after_point;
  return true;
}

// The shortest decimal that rounds to x (x > 0, finite), and among those of
// that length the one nearest to x: the decimal a shortest round-trip
// printer (such as Python's repr) produces.
Decimal shortest_decimal(double x) {
  char buf[64];
  for (int prec = 1; prec <= 17; ++prec) {
    std::snprintf(buf, sizeof buf, "%.*e", prec - 1, x);
    if (std::strtod(buf, nullptr) == x) {
      Decimal d{};
      parse_sci(buf, &d);
      return d;
    }
    // The nearest prec-digit decimal may fall just outside x's rounding
    // interval while its neighbour one unit above or below lies inside (the
    // interval is lopsided at powers of two). Try both, nearest first.
    Decimal r{};
    if (!parse_sci(buf, &r)) continue;
    Decimal best{};
    double best_dist = -1.0;
    for (int dir = -1; dir <= 1; dir += 2) {
      if (dir < 0 && r.mant == 0) continue;
      const uint64_t mm = r.mant + (uint64_t)(int64_t)dir;
      char cand[64];
      std::snprintf(cand, sizeof cand, "%llue%d", (unsigned long long)mm, r.exp10);
      const double v = std::strtod(cand, nullptr);
      if (v != x) continue;
      const long double dist = std::fabs((long double)mm * std::pow(10.0L, r.exp10) - (long double)x);
      if (best_dist < 0 || dist < best_dist) {
        best_dist = (double)dist;
        best = Decimal{mm, r.exp10};
      }
    }
    if (best_dist >= 0) return best;
  }
  Decimal d{};
  std::snprintf(buf, sizeof buf, "%.16e", x);
  parse_sci(buf, &d);
  return d;
}

// floor(n * x) (or ceil) for 0 <= n < 2^31 and x >= 0 read as its shortest
// decimal, exactly; results above INT32_MAX saturate there.
int64_t scaled_round(int64_t n, double x, bool ceil_it) {
  if (n <= 0 || !(x > 0.0)) return 0;
  if (!std::isfinite(x)) return INT32_MAX;
  const Decimal d = shortest_decimal(x);
  unsigned __int128 num = (unsigned __int128)n * d.mant;
  if (d.exp10 >= 0) {
    for (int i = 0; i < d.exp10 && num <= INT32_MAX; ++i) num *= 10;
    return num > INT32_MAX ? INT32_MAX : (int64_t)num;
  }
  // n * mant < 2^31 * 10^17 < 10^27: a divisor of 10^28 or more leaves 0.
  if (-d.exp10 >= 28) return ceil_it ? (num > 0 ? 1 : 0) : 0;
  unsigned __int128 den = 1;
  for (int i = 0; i < -d.exp10; ++i) den *= 10;
  const unsigned __int128 q = num / den + (ceil_it && num % den != 0 ? 1 : 0);
  return q > INT32_MAX ? INT32_MAX : (int64_t)q;
}

}  // namespace

int32_t f3c_ceil_ratio(int32_t steps, double rho) { return (int32_t)scaled_round(steps, rho, true); }

int32_t f3c_pcsc_quota(int32_t k, int32_t n_tokens, double sigma, double mu, int32_t k_anchor, double gamma_up) {
  const double bound = n_tokens - sigma * std::exp(mu * (k - k_anchor)) / gamma_up;
  const double f = std::floor(bound);
  if (!(f > 0)) return 0;
  if (f > n_tokens) return n_tokens;
  return (int32_t)f;
}

int32_t f3c_phase_quota(int32_t k, int32_t steps, int32_t n_tokens, int32_t n_cache_phase2, double rho_a,
                        double rho_off, double xi, int32_t f_corr) {
  if (k <= f3c_ceil_ratio(steps, rho_a)) return 0;
  const int32_t k_off = f3c_ceil_ratio(steps, rho_off);
  if (k < k_off) return n_cache_phase2;
  const int32_t k_refine = k - k_off;
  if (f_corr > 0 && (k_refine + 1) % f_corr == 0) return 0;
  return (int32_t)scaled_round(n_tokens, xi, false);
}

int32_t f3c_tau_forces_full(int32_t consecutive, int32_t tau, int32_t reading) {
  if (tau <= 0) return 0;
  return consecutive >= (reading == F3C_TAU_LITERAL ? tau : tau - 1);
}

int f3c_schedule_plan(const f3c_schedule_cfg* c, double sigma, int32_t* n_cache_out) {
  if (!c || !n_cache_out) return fail(F3C_EINVAL, "NULL argument");
  if (c->steps < 1 || c->n_tokens < 1) return fail(F3C_EINVAL, "need steps >= 1 and n_tokens >= 1");
  if (!std::isfinite(sigma) || !std::isfinite(c->mu) || !(c->gamma_up > 0) || !std::isfinite(c->gamma_up))
    return fail(F3C_EINVAL, "sigma and mu must be finite and gamma_up positive");
  if (!(c->rho_a >= 0 && c->rho_a <= 1) || !(c->rho_off >= 0 && c->rho_off <= 1) || !(c->xi >= 0 && c->xi <= 1))
    return fail(F3C_EINVAL, "rho_a, rho_off and xi must lie in [0, 1]");
  if (c->f_corr < 0 || c->tau < 0) return fail(F3C_EINVAL, "f_corr and tau must be >= 0");
  if (c->tau_reading != F3C_TAU_CYCLE && c->tau_reading != F3C_TAU_LITERAL) return fail(F3C_EINVAL, "bad tau_reading");
  const int32_t k_anchor = f3c_ceil_ratio(c->steps, c->rho_a);
  int32_t run = 0;                    // cached steps in a row before step k
  for (int32_t k = 1; k <= c->steps; ++k) {
    const int32_t phase2 = f3c_pcsc_quota(k, c->n_tokens, sigma, c->mu, k_anchor, c->gamma_up);
    int32_t n = f3c_phase_quota(k, c->steps, c->n_tokens, phase2, c->rho_a, c->rho_off, c->xi, c->f_corr);
    if (n > 0 && f3c_tau_forces_full(run, c->tau, c->tau_reading)) n = 0;
    run = n > 0 ? run + 1 : 0;
    n_cache_out[k - 1] = n;
  }
  return F3C_OK;
}

}  // extern "C"
