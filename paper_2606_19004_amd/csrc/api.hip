// C ABI of the denoise-step library: argument validation, workspace layout and
// the launch sequence of each entry point (see include/ditstep.h).
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <limits>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/ditstep.h"
#include "internal.h"
#include "host_checks.h"

using namespace dit;
using dit::set_error;

namespace {

#define HIP_TRY(expr)                                                                         \
  do {                                                                                        \
    hipError_t e_ = (expr);                                                                   \
    if (e_ != hipSuccess) return set_error(DIT_ERR_HIP, "%s failed: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// ---- opt-in kernel timing (dit_profile_begin / dit_profile_end) ----
struct ProfRec {
  const char* name;
  double flops, bytes;
  hipEvent_t a, b;
};
struct Prof {
  std::mutex mu;
  std::atomic<bool> on{false};   // read without the lock on every launch
  std::vector<ProfRec> recs;
};
Prof g_prof;

// set while an allocation-free entry point runs on this thread: no timing events are created
thread_local bool g_no_events = false;

#ifdef DITSTEP_DEBUG
// Debug builds: every launch is followed by a synchronisation of its stream (unless the stream is
// being captured) and a check of the launch and of the kernel's completion.
template <class F>
hipError_t checked(hipStream_t s, F&& launch) {
  hipError_t e = launch();
  if (e != hipSuccess) return e;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if ((e = hipStreamIsCapturing(s, &cs)) != hipSuccess) return e;
  if (cs != hipStreamCaptureStatusNone) return hipSuccess;
  if ((e = hipStreamSynchronize(s)) != hipSuccess) return e;
  return hipGetLastError();
}
#endif

template <class F>
hipError_t timed(const char* name, double flops, double bytes, hipStream_t s, F&& launch_) {
#ifdef DITSTEP_DEBUG
  auto launch = [&]() { return checked(s, launch_); };
#else
  auto& launch = launch_;
#endif
  if (g_no_events || !g_prof.on.load(std::memory_order_acquire)) return launch();
  hipEvent_t a, b;
  hipError_t e = hipEventCreate(&a);
  if (e != hipSuccess) return e;
  if ((e = hipEventCreate(&b)) != hipSuccess) return e;
  if ((e = hipEventRecord(a, s)) != hipSuccess) return e;
  hipError_t le = launch();
  if ((e = hipEventRecord(b, s)) != hipSuccess) return e;
  std::lock_guard<std::mutex> g(g_prof.mu);
  g_prof.recs.push_back(ProfRec{name, flops, bytes, a, b});
  return le;
}
#define TIMED(name, flops, bytes, s, expr) HIP_TRY(timed(name, (double)(flops), (double)(bytes), s, [&]() { return (expr); }))

double gemm_flops(const GemmPair& p) {
  double f = 0;
  for (int i = 0; i < p.nprob; i++) f += 2.0 * p.p[i].M * p.p[i].N * p.p[i].K;
  return f;
}

inline size_t al256(size_t x) { return (x + 255) & ~(size_t)255; }
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
inline size_t esize(int32_t dtype) { return dtype == DIT_BF16 ? 2 : 4; }
inline hipStream_t hs(dit_stream s) { return (hipStream_t)s; }

dit_status check_ws(void* ws, size_t have, size_t need) {
  if (need == 0) return DIT_OK;
  if (!ws) return set_error(DIT_ERR_WORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)ws & 255) return set_error(DIT_ERR_WORKSPACE, "workspace not 256-byte aligned");
  if (have < need) return set_error(DIT_ERR_WORKSPACE, "workspace %zu bytes < %zu needed", have, need);
  return DIT_OK;
}

// offsets into the block workspace
struct BlockWs {
  size_t mod, silu, xs, rope, h, qkv, u, total;
};
// scratch of the MFMA GEMV: 16 samples x K, as bf16 hi and lo parts
inline size_t xs_bytes(int64_t K) { return al256(2 * 16 * (size_t)K * 2); }
BlockWs block_layout(const dit_block_config* c, int64_t B) {
  BlockWs w;
  size_t es = esize(c->dtype);
  size_t S = (size_t)c->n_img + c->n_txt, D = c->hidden, F = c->mlp_hidden;
  size_t npos = std::max(c->grid_h, c->grid_w);
  size_t off = 0;
  w.mod = off;  off += al256(2 * B * 6 * D * 4);
  w.silu = off; off += al256(B * D * 4);
  w.xs = off;   off += xs_bytes(std::max<size_t>(D, 256));
  w.rope = off; off += al256(npos * (c->head_dim / 4) * 2 * 4);
  w.h = off;    off += al256(B * S * D * es);
  w.qkv = off;  off += al256(B * S * 3 * D * es);
  w.u = off;    off += al256(B * S * F * es);
  w.total = off;
  return w;
}

dit_status check_block_args(const dit_block_config* c, const dit_block_weights* w, int32_t batch,
                            const float* temb, void* x_img, void* x_txt) {
  dit_status st = check_config(c);
  if (st) return st;
  if (!w) return set_error(DIT_ERR_INVALID_ARG, "weights is NULL");
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch %d < 0", batch);
  if (batch == 0) return DIT_OK;
  if (!temb || !x_img || (c->n_txt > 0 && !x_txt)) return set_error(DIT_ERR_INVALID_ARG, "temb/x_img/x_txt NULL");
  if (!aligned16(temb) || !aligned16(x_img) || (x_txt && !aligned16(x_txt)))
    return set_error(DIT_ERR_INVALID_ARG, "temb/x_img/x_txt must be 16-byte aligned");
  for (int s = 0; s < 2; s++) {
    if (!w->mod_w[s] || !w->qkv_w[s] || !w->out_w[s] || !w->mlp1_w[s] || !w->mlp2_w[s])
      return set_error(DIT_ERR_INVALID_ARG, "a weight matrix of stream %d is NULL", s);
    const void* all[10] = {w->mod_w[s], w->mod_b[s], w->qkv_w[s], w->qkv_b[s], w->out_w[s],
                           w->out_b[s], w->mlp1_w[s], w->mlp1_b[s], w->mlp2_w[s], w->mlp2_b[s]};
    for (const void* p : all)
      if (p && ((uintptr_t)p & 7)) return set_error(DIT_ERR_INVALID_ARG, "weights must be 8-byte aligned");
  }
  // the MFMA GEMM addresses its A operand with 31-bit byte offsets, and row counts (B x S) are 32-bit
  // in both paths: the largest activation buffer stays below 2 GiB
  {
    double S = (double)c->n_img + c->n_txt;
    double big = (double)batch * S * std::max(3 * c->hidden, c->mlp_hidden) * (double)esize(c->dtype);
    if (big >= 2147483648.0) return set_error(DIT_ERR_UNSUPPORTED, "activation buffer of %.0f bytes exceeds 2 GiB", big);
  }
  return DIT_OK;
}

// One stream's slice of a joint [B][S][cols] buffer (text rows first).
RowMap joint_rows(const dit_block_config* c, int stream, int64_t cols) {
  int64_t S = (int64_t)c->n_img + c->n_txt;
  if (stream == 0) return RowMap{c->n_img, S * cols, cols, (int64_t)c->n_txt * cols};
  return RowMap{std::max(c->n_txt, 1), S * cols, cols, 0};
}
RowMap stream_rows(int64_t n, int64_t cols) { return RowMap{std::max<int64_t>(n, 1), n * cols, cols, 0}; }

// out = W act(in) + b with act = SiLU when silu_in: MFMA (hi/lo split) for bf16
// weights, VALU for fp32 weights (which first writes SiLU(in) to silu_buf)
dit_status run_gemv(const dit_block_config* c, GemvArgs g, bool silu_in, float* silu_buf, void* xs,
                    const char* name, hipStream_t s) {
  double flops = 2.0 * g.nstreams * g.B * (double)g.N * g.K;
  double bytes = (double)g.nstreams * g.N * (double)g.K * esize(c->dtype);
  if (c->dtype == DIT_BF16) {
    TIMED(name, flops, bytes, s, gemv_bf16(g, (u16*)xs, silu_in ? 1 : 0, s));
    return DIT_OK;
  }
  if (silu_in) {
    TIMED("small_elementwise", 0, (double)g.B * g.K * 8, s, silu_f32(g.in, silu_buf, (int64_t)g.B * g.in_bstride, s));
    g.in = silu_buf;
  }
  TIMED(name, flops, bytes, s, gemv(g, c->dtype, s));
  return DIT_OK;
}

// mod[s][b][6D] = W_mod[s] SiLU(temb[b]) + b_mod[s]
dit_status run_modulation(const dit_block_config* c, const dit_block_weights* w, int B, const float* temb,
                          char* ws, const BlockWs& L, hipStream_t s) {
  const int D = c->hidden;
  float* mod = (float*)(ws + L.mod);
  GemvArgs g{};
  for (int st = 0; st < 2; st++) {
    g.W[st] = w->mod_w[st];
    g.bias[st] = w->mod_b[st];
    g.out[st] = mod + (size_t)st * B * 6 * D;
  }
  g.out_bstride = 6 * D;
  g.in = temb;
  g.in_bstride = D;
  g.N = 6 * D;
  g.K = D;
  g.B = B;
  g.nstreams = 2;
  return run_gemv(c, g, true, (float*)(ws + L.silu), ws + L.xs, "mod_gemv", s);
}

// The modulation depends only on the timestep embedding, which every block of a step shares, so the
// step computes it for up to MOD_GROUP blocks in one GEMV launch (2 weight slots per block):
// dst + i * 2 B 6D holds block i's mod[s][b][6D], laid out as in run_modulation.
constexpr int MOD_GROUP = GEMV_SLOTS / 2;
dit_status run_modulation_group(const dit_block_config* c, const dit_block_weights* blocks, int n, int B,
                                const float* temb, float* dst, char* ws, const BlockWs& L, hipStream_t s) {
  const int D = c->hidden;
  GemvArgs g{};
  for (int i = 0; i < n; i++)
    for (int st = 0; st < 2; st++) {
      g.W[2 * i + st] = blocks[i].mod_w[st];
      g.bias[2 * i + st] = blocks[i].mod_b[st];
      g.out[2 * i + st] = dst + ((size_t)2 * i + st) * B * 6 * D;
    }
  g.out_bstride = 6 * D;
  g.in = temb;
  g.in_bstride = D;
  g.N = 6 * D;
  g.K = D;
  g.B = B;
  g.nstreams = 2 * n;
  return run_gemv(c, g, true, (float*)(ws + L.silu), ws + L.xs, "mod_gemv", s);
}

// h = LN(x)(1+scale)+shift for both streams into the joint [B][S][D] buffer
#ifdef DITSTEP_DEBUG
// Debug builds: the entry points of the block path register the buffers whose sizes they know (the
// workspace, the residual streams, the modulation, the block's weights), and every operand range a
// GEMM, attention or LayerNorm launch addresses must lie inside one of them.
struct DbgRegions {
  const char* base[32];
  size_t bytes[32];
  int n = 0;
  void add(const void* p, size_t b) {
    if (p && n < 32) {
      base[n] = (const char*)p;
      bytes[n] = b;
      n++;
    }
  }
  bool holds(const void* p, size_t b) const {
    const char* q = (const char*)p;
    for (int i = 0; i < n; i++)
      if (q >= base[i] && q + b <= base[i] + bytes[i]) return true;
    return false;
  }
};
thread_local const DbgRegions* g_dbg = nullptr;
struct DbgScope {
  const DbgRegions* prev;
  explicit DbgScope(const DbgRegions* r) : prev(g_dbg) { g_dbg = r; }
  ~DbgScope() { g_dbg = prev; }
};
// one past the largest element a row map addresses for rows x cols (row maps grow with the row)
size_t map_extent(const RowMap& m, int64_t rows, int64_t cols) {
  return rows <= 0 ? 0 : (size_t)(row_offset(m, rows - 1) + cols);
}
DbgRegions block_regions(const dit_block_config* c, const dit_block_weights* w, int B, const void* x_img,
                         const void* x_txt, const char* ws, size_t ws_bytes, const float* mod) {
  DbgRegions r;
  const size_t es = esize(c->dtype), D = c->hidden, F = c->mlp_hidden;
  // test hook: register the workspace 4 KB short, so that the checks must refuse the launches
  // whose operands reach its end (the MLP hidden buffer is its last region)
  if (std::getenv("DITSTEP_DEBUG_SHRINK_WS") && ws_bytes > 4096) ws_bytes -= 4096;
  r.add(ws, ws_bytes);
  r.add(x_img, (size_t)B * c->n_img * D * es);
  r.add(x_txt, (size_t)B * c->n_txt * D * es);
  r.add(mod, (size_t)2 * B * 6 * D * 4);
  for (int i = 0; i < 2; i++) {
    r.add(w->mod_w[i], 6 * D * D * es);
    r.add(w->mod_b[i], 6 * D * es);
    r.add(w->qkv_w[i], 3 * D * D * es);
    r.add(w->qkv_b[i], 3 * D * es);
    r.add(w->out_w[i], D * D * es);
    r.add(w->out_b[i], D * es);
    r.add(w->mlp1_w[i], F * D * es);
    r.add(w->mlp1_b[i], F * es);
    r.add(w->mlp2_w[i], D * F * es);
    r.add(w->mlp2_b[i], D * es);
  }
  return r;
}
dit_status dbg_fail(const char* what, const char* operand, int i) {
  return set_error(DIT_ERR_INVALID_ARG, "debug check: %s launch, problem %d: %s outside every known buffer", what,
                   i, operand);
}
dit_status dbg_gemm(const GemmPair& pr, size_t es, const char* what) {
  if (!g_dbg) return DIT_OK;
  for (int i = 0; i < pr.nprob; i++) {
    const GemmProblem& p = pr.p[i];
    if (p.M <= 0 || p.N <= 0) continue;
    if (!g_dbg->holds(p.A, map_extent(p.amap, p.M, p.K) * es)) return dbg_fail(what, "A", i);
    if (!g_dbg->holds(p.W, (size_t)p.N * p.K * es)) return dbg_fail(what, "W", i);
    if (p.bias && !g_dbg->holds(p.bias, (size_t)p.N * es)) return dbg_fail(what, "bias", i);
    if (!g_dbg->holds(p.C, map_extent(p.cmap, p.M, p.N) * es)) return dbg_fail(what, "C", i);
    if (p.gate) {
      const int64_t nb = (p.M - 1) / p.cmap.rows_per_batch + 1;
      if (!g_dbg->holds(p.gate, (size_t)((nb - 1) * p.gate_bstride + p.N) * 4)) return dbg_fail(what, "gate", i);
    }
  }
  return DIT_OK;
}
dit_status dbg_attn(const AttnArgs& a, size_t es) {
  if (!g_dbg) return DIT_OK;
  const size_t in = (size_t)((a.B - 1) * a.qs_b + (a.S - 1) * a.qs_s + (a.H - 1) * a.qs_h + a.d) * es;
  const size_t out = (size_t)((a.B - 1) * a.os_b + (a.S - 1) * a.os_s + (a.H - 1) * a.os_h + a.d) * es;
  if (!g_dbg->holds(a.q, in)) return dbg_fail("attention", "q", 0);
  if (!g_dbg->holds(a.k, in)) return dbg_fail("attention", "k", 0);
  if (!g_dbg->holds(a.v, in)) return dbg_fail("attention", "v", 0);
  if (!g_dbg->holds(a.o, out)) return dbg_fail("attention", "o", 0);
  return DIT_OK;
}
dit_status dbg_ln(const LnArgs& a, size_t es) {
  if (!g_dbg) return DIT_OK;
  for (int i = 0; i < 2; i++) {
    if (a.rows[i] <= 0) continue;
    if (!g_dbg->holds(a.x[i], map_extent(a.xmap[i], a.rows[i], a.D) * es)) return dbg_fail("ln_modulate", "x", i);
    if (!g_dbg->holds(a.out, map_extent(a.omap[i], a.rows[i], a.D) * es)) return dbg_fail("ln_modulate", "out", i);
    const int64_t nb = (a.rows[i] - 1) / a.xmap[i].rows_per_batch + 1;
    const size_t mod = (size_t)((nb - 1) * a.mod_bstride + std::max(a.shift_off, a.scale_off) + a.D) * 4;
    if (!g_dbg->holds(a.mod[i], mod)) return dbg_fail("ln_modulate", "mod", i);
  }
  return DIT_OK;
}
#define DBG_CHECK(expr)                      \
  do {                                       \
    if (dit_status d_ = (expr)) return d_;   \
  } while (0)
#else
#define DBG_CHECK(expr) \
  do {                  \
  } while (0)
#endif

dit_status run_ln(const dit_block_config* c, int B, const void* x_img, const void* x_txt, const float* mod,
                  char* ws, const BlockWs& L, int shift_off, int scale_off, hipStream_t s) {
  const int D = c->hidden;
  LnArgs a{};
  a.x[0] = x_img;
  a.x[1] = x_txt;
  a.xmap[0] = stream_rows(c->n_img, D);
  a.xmap[1] = stream_rows(c->n_txt, D);
  a.out = ws + L.h;
  a.omap[0] = joint_rows(c, 0, D);
  a.omap[1] = joint_rows(c, 1, D);
  a.mod[0] = mod;
  a.mod[1] = mod + (size_t)B * 6 * D;
  a.mod_bstride = 6 * D;
  a.shift_off = shift_off;
  a.scale_off = scale_off;
  a.rows[0] = (int64_t)B * c->n_img;
  a.rows[1] = (int64_t)B * c->n_txt;
  a.D = D;
  a.eps = c->ln_eps;
  DBG_CHECK(dbg_ln(a, esize(c->dtype)));
  TIMED("ln_modulate", 0, 2.0 * (a.rows[0] + a.rows[1]) * D * esize(c->dtype), s, ln_modulate(a, c->dtype, s));
  return DIT_OK;
}

GemmProblem problem(const void* A, RowMap am, const void* W, const void* bias, void* C, RowMap cm, int M, int N, int K) {
  GemmProblem p{};
  p.A = A;
  p.amap = am;
  p.W = W;
  p.bias = bias;
  p.C = C;
  p.cmap = cm;
  p.M = M;
  p.N = N;
  p.K = K;
  return p;
}

// the MLP half: h2 = LN(x)(1+scale2)+shift2; u = GELU(W1 h2 + b1); x += gate2 (W2 u + b2)
dit_status run_mlp_half(const dit_block_config* c, const dit_block_weights* w, int B, void* x_img, void* x_txt,
                        const float* mod, char* ws, const BlockWs& L, hipStream_t s) {
  const int D = c->hidden, F = c->mlp_hidden;
  const int rows[2] = {B * c->n_img, B * c->n_txt};
  void* x[2] = {x_img, x_txt};
  const int64_t nstream[2] = {c->n_img, c->n_txt};
  dit_status st = run_ln(c, B, x_img, x_txt, mod, ws, L, 3 * D, 4 * D, s);
  if (st) return st;
  GemmPair up{}, down{};
  up.nprob = down.nprob = 2;
  for (int i = 0; i < 2; i++) {
    up.p[i] = problem(ws + L.h, joint_rows(c, i, D), w->mlp1_w[i], w->mlp1_b[i], ws + L.u, joint_rows(c, i, F),
                      rows[i], F, D);
    down.p[i] = problem(ws + L.u, joint_rows(c, i, F), w->mlp2_w[i], w->mlp2_b[i], x[i], stream_rows(nstream[i], D),
                        rows[i], D, F);
    down.p[i].gate = mod + (size_t)i * B * 6 * D + 5 * D;
    down.p[i].gate_bstride = 6 * D;
  }
  DBG_CHECK(dbg_gemm(up, esize(c->dtype), "gemm_mlp_up_gelu"));
  DBG_CHECK(dbg_gemm(down, esize(c->dtype), "gemm_mlp_down_gate"));
  TIMED("gemm_mlp_up_gelu", gemm_flops(up), 0, s, gemm(up, EPI_GELU, c->dtype, false, s));
  TIMED("gemm_mlp_down_gate", gemm_flops(down), 0, s, gemm(down, EPI_RESID, c->dtype, false, s));
  return DIT_OK;
}

struct StepWs {
  size_t temb, ximg, xtxt, v, mods, inner, total;
};

size_t timestep_ws(const dit_block_config* c, int64_t B) {
  return al256(B * 256 * 4) + 2 * al256(B * c->hidden * 4) + xs_bytes(std::max(c->hidden, 256));
}
size_t patch_ws(const dit_block_config* c, int64_t B, int C) {
  return c->dtype == DIT_BF16 ? al256(B * c->n_img * C * 2) : 0;
}
size_t final_ws(const dit_block_config* c, int64_t B) {
  return al256(B * c->hidden * 4) + al256(B * 2 * c->hidden * 4) + al256(B * c->n_img * c->hidden * esize(c->dtype)) +
         xs_bytes(c->hidden);
}

StepWs step_layout(const dit_block_config* c, int64_t B, int C) {
  StepWs w;
  size_t es = esize(c->dtype);
  size_t off = 0;
  w.temb = off; off += al256(B * c->hidden * 4);
  w.ximg = off; off += al256(B * c->n_img * c->hidden * es);
  w.xtxt = off; off += al256(B * c->n_txt * c->hidden * es);
  w.v = off;    off += al256(B * c->n_img * C * 4);
  w.mods = off; off += al256((size_t)MOD_GROUP * 2 * B * 6 * c->hidden * 4);
  w.inner = off;
  size_t inner = std::max({block_layout(c, B).total, timestep_ws(c, B), patch_ws(c, B, C), final_ws(c, B)});
  w.total = off + inner;
  return w;
}

dit_status check_step_weights(const dit_step_weights* w) {
  if (!w) return set_error(DIT_ERR_INVALID_ARG, "step weights NULL");
  if (!w->t1_w || !w->t2_w || !w->in_w || !w->fmod_w || !w->fout_w)
    return set_error(DIT_ERR_INVALID_ARG, "a step weight matrix is NULL");
  return DIT_OK;
}

dit_status run_timestep(const dit_block_config* c, const dit_step_weights* w, int B, const float* t_dev, float t,
                        float* temb, char* ws, hipStream_t s) {
  const int D = c->hidden;
  float* e = (float*)ws;
  float* h1 = (float*)(ws + al256((size_t)B * 256 * 4));
  float* s1 = (float*)(ws + al256((size_t)B * 256 * 4) + al256((size_t)B * D * 4));
  char* xs = ws + al256((size_t)B * 256 * 4) + 2 * al256((size_t)B * D * 4);
  TIMED("small_elementwise", 0, (double)B * 256 * 4, s, timestep_sinusoid(t_dev, t, e, B, s));
  GemvArgs g{};
  g.W[0] = w->t1_w;
  g.bias[0] = w->t1_b;
  g.out[0] = h1;
  g.out_bstride = D;
  g.in = e;
  g.in_bstride = 256;
  g.N = D;
  g.K = 256;
  g.B = B;
  g.nstreams = 1;
  dit_status st = run_gemv(c, g, false, nullptr, xs, "timestep_gemv", s);
  if (st) return st;
  g.W[0] = w->t2_w;
  g.bias[0] = w->t2_b;
  g.out[0] = temb;
  g.in = h1;
  g.in_bstride = D;
  g.K = D;
  return run_gemv(c, g, true, s1, xs, "timestep_gemv", s);
}

dit_status run_patch(const dit_block_config* c, const dit_step_weights* w, int B, int C, const float* latent,
                     void* x_img, char* ws, hipStream_t s) {
  const int D = c->hidden;
  const int M = B * c->n_img;
  const void* A = latent;
  if (c->dtype == DIT_BF16) {
    TIMED("small_elementwise", 0, (double)M * C * 6, s, cast_f32_to_bf16(latent, (u16*)ws, (int64_t)M * C, s));
    A = ws;
  }
  GemmPair p{};
  p.nprob = 1;
  p.p[0] = problem(A, contiguous_rows(C), w->in_w, w->in_b, x_img, contiguous_rows(D), M, D, C);
  TIMED("gemm_patch_embed", gemm_flops(p), 0, s, gemm(p, EPI_STORE, c->dtype, false, s));
  return DIT_OK;
}

dit_status run_final(const dit_block_config* c, const dit_step_weights* w, int B, int C, const float* temb,
                     const void* x_img, float* v, char* ws, hipStream_t s) {
  const int D = c->hidden;
  float* s1 = (float*)ws;
  float* fm = (float*)(ws + al256((size_t)B * D * 4));
  char* h = ws + al256((size_t)B * D * 4) + al256((size_t)B * 2 * D * 4);
  char* xs = h + al256((size_t)B * c->n_img * D * esize(c->dtype));
  GemvArgs g{};
  g.W[0] = w->fmod_w;
  g.bias[0] = w->fmod_b;
  g.out[0] = fm;
  g.out_bstride = 2 * D;
  g.in = temb;
  g.in_bstride = D;
  g.N = 2 * D;
  g.K = D;
  g.B = B;
  g.nstreams = 1;
  dit_status st = run_gemv(c, g, true, s1, xs, "final_gemv", s);
  if (st) return st;
  LnArgs a{};
  a.x[0] = x_img;
  a.xmap[0] = stream_rows(c->n_img, D);
  a.out = h;
  a.omap[0] = stream_rows(c->n_img, D);
  a.mod[0] = fm;
  a.mod_bstride = 2 * D;
  a.shift_off = 0;
  a.scale_off = D;
  a.rows[0] = (int64_t)B * c->n_img;
  a.rows[1] = 0;
  a.D = D;
  a.eps = c->ln_eps;
  TIMED("ln_modulate", 0, 2.0 * a.rows[0] * D * esize(c->dtype), s, ln_modulate(a, c->dtype, s));
  GemmPair p{};
  p.nprob = 1;
  p.p[0] = problem(h, contiguous_rows(D), w->fout_w, w->fout_b, v, contiguous_rows(C), B * c->n_img, C, D);
  TIMED("gemm_final", gemm_flops(p), 0, s, gemm(p, EPI_STORE, c->dtype, true, s));
  return DIT_OK;
}

// ---- fixed device scratch of the allocation-free timestep embedding ----
// The array lives in the library's code object, one copy per GPU it runs on, for the life of the
// process. Host code never uses its name as an address (on the host it is only a stand-in): the
// device address comes from hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kTimestepScratchBytes = DIT_TIMESTEP_SCRATCH_BYTES;
}  // namespace
static __device__ __align__(256) char scratch[DIT_TIMESTEP_SCRATCH_BYTES];
namespace {

struct ScratchAddrs {
  std::mutex mu;
  void* ptr[64] = {};
};
ScratchAddrs g_scratch;

dit_status timestep_scratch(void** out) {
  int dev = -1;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return set_error(DIT_ERR_UNSUPPORTED, "device %d: at most 64 devices", dev);
  std::lock_guard<std::mutex> g(g_scratch.mu);
  if (!g_scratch.ptr[dev]) {
    void* p = nullptr;
    hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return set_error(DIT_ERR_HIP, "hipGetSymbolAddress(scratch) failed on device %d: %s", dev, hipGetErrorString(e));
    g_scratch.ptr[dev] = p;
  }
  *out = g_scratch.ptr[dev];
  return DIT_OK;
}

}  // namespace

// ===========================================================================
// exported entry points
// ===========================================================================
extern "C" {

size_t dit_block_workspace_bytes(const dit_block_config* cfg, int32_t batch) {
  if (check_config(cfg) != DIT_OK || batch < 0) return 0;
  return block_layout(cfg, batch).total;
}

}  // extern "C"

namespace {
// One block on checked arguments. mod_pre: the block's modulation computed beforehand (layout of
// run_modulation), or null to compute it here into the workspace. rope_ready: the workspace already
// holds the RoPE table (it depends only on the grid and head size, so a stack of blocks on one
// workspace fills it once).
dit_status block_body(const dit_block_config* c, const dit_block_weights* w, int B, const float* temb, void* x_img,
                      void* x_txt, char* ws, const BlockWs& L, const float* mod_pre, bool rope_ready, hipStream_t s) {
  dit_status st = DIT_OK;
  const int D = c->hidden, d = c->head_dim, H = c->heads;
  const int S = c->n_img + c->n_txt;
  const int rows[2] = {B * c->n_img, B * c->n_txt};
  void* x[2] = {x_img, x_txt};
  const int64_t nstream[2] = {c->n_img, c->n_txt};
  const float* mod = mod_pre ? mod_pre : (const float*)(ws + L.mod);
  float* rope = (float*)(ws + L.rope);
#ifdef DITSTEP_DEBUG
  const DbgRegions dbg_r = block_regions(c, w, B, x_img, x_txt, ws, L.total, mod);
  const DbgScope dbg_scope(&dbg_r);
#endif

  if (!mod_pre && (st = run_modulation(c, w, B, temb, ws, L, s))) return st;
  if (c->rope && !rope_ready)
    TIMED("small_elementwise", 0, 0, s, rope_table(rope, std::max(c->grid_h, c->grid_w), d, c->rope_theta, s));
  // pre-attention LN + modulate into h
  if ((st = run_ln(c, B, x_img, x_txt, mod, ws, L, 0, D, s))) return st;
  // QKV projection straight into the joint [B][S][3][H][d] buffer (+ RoPE on image q, k)
  GemmPair qkv{};
  qkv.nprob = 2;
  for (int i = 0; i < 2; i++) {
    qkv.p[i] = problem(ws + L.h, joint_rows(c, i, D), w->qkv_w[i], w->qkv_b[i], ws + L.qkv, joint_rows(c, i, 3 * D),
                       rows[i], 3 * D, D);
    qkv.p[i].head_dim = d;
    qkv.p[i].hidden = D;
    qkv.p[i].grid_w = c->grid_w;
  }
  if (c->rope) {
    qkv.p[0].rope_tab = rope;
    qkv.p[0].rope_npos = std::max(c->grid_h, c->grid_w);
  }
  DBG_CHECK(dbg_gemm(qkv, esize(c->dtype), "gemm_qkv_rope"));
  TIMED("gemm_qkv_rope", gemm_flops(qkv), 0, s, gemm(qkv, EPI_QKV, c->dtype, false, s));
  // joint attention over [text ; image]; output o reuses the h buffer
  AttnArgs at{};
  char* qkvp = ws + L.qkv;
  size_t es = esize(c->dtype);
  at.q = qkvp;
  at.k = qkvp + (size_t)D * es;
  at.v = qkvp + (size_t)2 * D * es;
  at.o = ws + L.h;
  at.B = B;
  at.H = H;
  at.S = S;
  at.d = d;
  at.qs_b = (int64_t)S * 3 * D;
  at.qs_s = 3 * D;
  at.qs_h = d;
  at.os_b = (int64_t)S * D;
  at.os_s = D;
  at.os_h = d;
  at.scale = 1.0f / std::sqrt((float)d);
  DBG_CHECK(dbg_attn(at, esize(c->dtype)));
  TIMED("attention", 4.0 * B * H * (double)S * S * d, 0, s, attention(at, c->dtype, s));
  // output projection + gate1 residual, in place on x
  GemmPair proj{};
  proj.nprob = 2;
  for (int i = 0; i < 2; i++) {
    proj.p[i] = problem(ws + L.h, joint_rows(c, i, D), w->out_w[i], w->out_b[i], x[i], stream_rows(nstream[i], D),
                        rows[i], D, D);
    proj.p[i].gate = mod + (size_t)i * B * 6 * D + 2 * D;
    proj.p[i].gate_bstride = 6 * D;
  }
  DBG_CHECK(dbg_gemm(proj, esize(c->dtype), "gemm_out_gate"));
  TIMED("gemm_out_gate", gemm_flops(proj), 0, s, gemm(proj, EPI_RESID, c->dtype, false, s));
  return run_mlp_half(c, w, B, x_img, x_txt, mod, ws, L, s);
}

// Blocks [0, n) in order on the block workspace `inner`; their modulation is computed MOD_GROUP
// blocks at a time into mods (first_ready: the first group's is there already).
dit_status run_blocks(const dit_block_config* c, const dit_block_weights* blocks, int n, int B, const float* temb,
                      void* ximg, void* xtxt, float* mods, char* inner, const BlockWs& BL, bool first_ready,
                      hipStream_t s) {
  dit_status st = DIT_OK;
  const size_t per = (size_t)2 * B * 6 * c->hidden;
  for (int g0 = 0; g0 < n; g0 += MOD_GROUP) {
    const int gn = std::min(MOD_GROUP, n - g0);
    if (!(g0 == 0 && first_ready) && (st = run_modulation_group(c, blocks + g0, gn, B, temb, mods, inner, BL, s)))
      return st;
    for (int i = 0; i < gn; i++)
      if ((st = block_body(c, &blocks[g0 + i], B, temb, ximg, xtxt, inner, BL, mods + i * per, g0 + i > 0, s)))
        return st;
  }
  return DIT_OK;
}
}  // namespace

extern "C" {

dit_status dit_block_forward(const dit_block_config* c, const dit_block_weights* w, int32_t batch, const float* temb,
                             void* x_img, void* x_txt, void* workspace, size_t workspace_bytes, dit_stream stream) {
  dit_status st = check_block_args(c, w, batch, temb, x_img, x_txt);
  if (st || batch == 0) return st;
  BlockWs L = block_layout(c, batch);
  if ((st = check_ws(workspace, workspace_bytes, L.total))) return st;
  return block_body(c, w, batch, temb, x_img, x_txt, (char*)workspace, L, nullptr, false, hs(stream));
}

dit_status dit_block_mlp(const dit_block_config* c, const dit_block_weights* w, int32_t batch, const float* temb,
                         void* x_img, void* x_txt, void* workspace, size_t workspace_bytes, dit_stream stream) {
  dit_status st = check_block_args(c, w, batch, temb, x_img, x_txt);
  if (st || batch == 0) return st;
  BlockWs L = block_layout(c, batch);
  if ((st = check_ws(workspace, workspace_bytes, L.total))) return st;
  char* ws = (char*)workspace;
  if ((st = run_modulation(c, w, batch, temb, ws, L, hs(stream)))) return st;
#ifdef DITSTEP_DEBUG
  const DbgRegions dbg_r = block_regions(c, w, batch, x_img, x_txt, ws, L.total, (const float*)(ws + L.mod));
  const DbgScope dbg_scope(&dbg_r);
#endif
  return run_mlp_half(c, w, batch, x_img, x_txt, (const float*)(ws + L.mod), ws, L, hs(stream));
}

dit_status joint_attention(const void* q, const void* k, const void* v, void* o, int32_t batch, int32_t heads,
                           int32_t seq, int32_t head_dim, int64_t qkv_stride_b, int64_t qkv_stride_s,
                           int64_t qkv_stride_h, int64_t o_stride_b, int64_t o_stride_s, int64_t o_stride_h,
                           float scale, int32_t dtype, dit_stream stream) {
  if (dtype != DIT_F32 && dtype != DIT_BF16) return set_error(DIT_ERR_INVALID_ARG, "dtype %d invalid", dtype);
  if (batch < 0 || heads < 0 || seq < 0) return set_error(DIT_ERR_INVALID_ARG, "negative size");
  if (head_dim != 64 && head_dim != 128) return set_error(DIT_ERR_UNSUPPORTED, "head_dim %d (64 or 128)", head_dim);
  if ((int64_t)batch * heads * seq == 0) return DIT_OK;
  if (!q || !k || !v || !o) return set_error(DIT_ERR_INVALID_ARG, "q/k/v/o NULL");
  if (!std::isfinite(scale)) return set_error(DIT_ERR_INVALID_ARG, "scale not finite");
  size_t es = esize(dtype);
  const int64_t strides[6] = {qkv_stride_b, qkv_stride_s, qkv_stride_h, o_stride_b, o_stride_s, o_stride_h};
  for (int64_t st : strides)
    if (st < 0 || (st * (int64_t)es) % 16) return set_error(DIT_ERR_INVALID_ARG, "strides must be >= 0 and keep 16-byte rows");
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o))
    return set_error(DIT_ERR_INVALID_ARG, "q/k/v/o must be 16-byte aligned");
  // the bf16 kernel addresses the keys of one (sample, head) with 31-bit byte offsets
  if (dtype == DIT_BF16 && (double)seq * qkv_stride_s * 2.0 >= 2147483648.0)
    return set_error(DIT_ERR_UNSUPPORTED, "seq * qkv_stride_s spans more than 2 GiB");
  AttnArgs a{};
  a.q = q;
  a.k = k;
  a.v = v;
  a.o = o;
  a.B = batch;
  a.H = heads;
  a.S = seq;
  a.d = head_dim;
  a.qs_b = qkv_stride_b;
  a.qs_s = qkv_stride_s;
  a.qs_h = qkv_stride_h;
  a.os_b = o_stride_b;
  a.os_s = o_stride_s;
  a.os_h = o_stride_h;
  a.scale = scale;
  TIMED("attention", 4.0 * batch * heads * (double)seq * seq * head_dim, 0, hs(stream), attention(a, dtype, hs(stream)));
  return DIT_OK;
}

dit_status flow_step(float* x, const float* v, const float* noise, int64_t n, float t, float t_next,
                     float noise_level, dit_stream stream) {
  if (n < 0) return set_error(DIT_ERR_INVALID_ARG, "n %lld < 0", (long long)n);
  float cx, cv, ce;
  dit_status st = flow_coefficients(t, t_next, noise_level, noise != nullptr, &cx, &cv, &ce);
  if (st) return st;
  if (n == 0) return DIT_OK;
  if (!x || !v) return set_error(DIT_ERR_INVALID_ARG, "x/v NULL");
  TIMED("flow_step", 0, (noise_level > 0.f ? 16.0 : 12.0) * n, hs(stream), flow_update(x, v, noise_level > 0.f ? noise : nullptr, n, cx, cv, ce, hs(stream)));
  return DIT_OK;
}

dit_status flow_logprob(const float* x, const float* v, const float* x_next, int32_t batch, int64_t n_per_sample,
                        float t, float t_next, float noise_level, double* logp, dit_stream stream) {
  if (batch < 0 || n_per_sample < 0)
    return set_error(DIT_ERR_INVALID_ARG, "batch %d / n_per_sample %lld < 0", batch, (long long)n_per_sample);
  if (!(noise_level > 0.f) || !std::isfinite(noise_level))
    return set_error(DIT_ERR_DOMAIN, "flow_logprob needs a finite noise_level > 0 (the ODE step has no density)");
  if (!(t > 0.f && t < 1.f) || !std::isfinite(t_next) || !(t_next < t))
    return set_error(DIT_ERR_DOMAIN, "flow_logprob needs 0 < t < 1 and t_next < t (t=%g, t_next=%g)", t, t_next);
  if (batch == 0) return DIT_OK;
  if (!logp) return set_error(DIT_ERR_INVALID_ARG, "logp NULL");
  if (n_per_sample > 0 && (!x || !v || !x_next)) return set_error(DIT_ERR_INVALID_ARG, "x/v/x_next NULL");
  const double td = t, h = (double)t_next - td, a = noise_level;
  const double var = a * a * td / (1.0 - td) * (-h);
  const double k1 = 0.5 * a * a / (1.0 - td);           // sigma^2 / (2t)
  const double cst = -0.5 * (double)n_per_sample * std::log(2.0 * M_PI * var);
  TIMED("flow_logprob", 0, 12.0 * batch * n_per_sample, hs(stream),
        flow_logprob_launch(x, v, x_next, batch, n_per_sample, h, k1, 1.0 - td, 0.5 / var, cst, logp, hs(stream)));
  return DIT_OK;
}

dit_status group_reward_stats(const float* rewards, int32_t groups, int32_t n, float adv_eps, int32_t k_select,
                              float* mean, float* stdv, float* adv, int32_t* order, int32_t* selected,
                              dit_stream stream) {
  if (groups < 0) return set_error(DIT_ERR_INVALID_ARG, "groups %d < 0", groups);
  if (n < 1 || n > 4096) return set_error(DIT_ERR_INVALID_ARG, "n %d outside [1, 4096]", n);
  if (k_select < 0 || k_select > n) return set_error(DIT_ERR_INVALID_ARG, "k_select %d outside [0, n=%d]", k_select, n);
  if (!(adv_eps >= 0.f) || !std::isfinite(adv_eps)) return set_error(DIT_ERR_INVALID_ARG, "adv_eps must be >= 0");
  if (groups == 0) return DIT_OK;
  if (!rewards) return set_error(DIT_ERR_INVALID_ARG, "rewards NULL");
  hipStream_t s = hs(stream);
  // NaN / Inf check on a host copy of the (small) input, before anything is written
  std::vector<float> host((size_t)groups * n);
  HIP_TRY(hipMemcpyAsync(host.data(), rewards, host.size() * 4, hipMemcpyDeviceToHost, s));
  HIP_TRY(hipStreamSynchronize(s));
  for (size_t i = 0; i < host.size(); i++)
    if (!std::isfinite(host[i])) return set_error(DIT_ERR_NAN, "reward %zu (group %zu) is not finite", i % n, i / n);
  TIMED("reward_stats", 0, 4.0 * groups * n, s, reward_stats(rewards, groups, n, adv_eps, k_select, mean, stdv, adv, order, selected, nullptr, DIT_ERR_NAN, s));
  return DIT_OK;
}

dit_status group_reward_stats_async(const float* rewards, int32_t groups, int32_t n, float adv_eps, int32_t k_select,
                                    float* mean, float* stdv, float* adv, int32_t* order, int32_t* selected,
                                    int32_t* status, dit_stream stream) {
  if (groups < 0) return set_error(DIT_ERR_INVALID_ARG, "groups %d < 0", groups);
  if (n < 1 || n > 4096) return set_error(DIT_ERR_INVALID_ARG, "n %d outside [1, 4096]", n);
  if (k_select < 0 || k_select > n) return set_error(DIT_ERR_INVALID_ARG, "k_select %d outside [0, n=%d]", k_select, n);
  if (!(adv_eps >= 0.f) || !std::isfinite(adv_eps)) return set_error(DIT_ERR_INVALID_ARG, "adv_eps must be >= 0");
  if (!status) return set_error(DIT_ERR_INVALID_ARG, "status NULL");
  if (groups == 0) return DIT_OK;
  if (!rewards) return set_error(DIT_ERR_INVALID_ARG, "rewards NULL");
  hipStream_t s = hs(stream);
  TIMED("reward_stats", 0, 4.0 * groups * n, s, reward_stats(rewards, groups, n, adv_eps, k_select, mean, stdv, adv, order, selected, status, DIT_ERR_NAN, s));
  return DIT_OK;
}

dit_status dit_timestep_embed(const dit_block_config* c, const dit_step_weights* w, int32_t batch, const float* t,
                              float* temb, void* workspace, size_t workspace_bytes, dit_stream stream) {
  dit_status st = check_config(c);
  if (st || (st = check_step_weights(w))) return st;
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch < 0");
  if (batch == 0) return DIT_OK;
  if (!t || !temb) return set_error(DIT_ERR_INVALID_ARG, "t/temb NULL");
  if ((st = check_ws(workspace, workspace_bytes, timestep_ws(c, batch)))) return st;
  return run_timestep(c, w, batch, t, 0.f, temb, (char*)workspace, hs(stream));
}

dit_status dit_timestep_embed_noalloc(const dit_block_config* c, const dit_step_weights* w, int32_t batch,
                                      const float* t, float* temb, dit_stream stream) {
  dit_status st = check_config(c);
  if (st || (st = check_step_weights(w))) return st;
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch < 0");
  if (batch == 0) return DIT_OK;
  if (!t || !temb) return set_error(DIT_ERR_INVALID_ARG, "t/temb NULL");
  const size_t need = timestep_ws(c, batch);
  if (need > kTimestepScratchBytes)
    return set_error(DIT_ERR_UNSUPPORTED, "batch %d at hidden %d needs %zu bytes of scratch, more than the %zu-byte device array",
                     batch, c->hidden, need, kTimestepScratchBytes);
  void* ws = nullptr;
  if ((st = timestep_scratch(&ws))) return st;
  g_no_events = true;
  st = run_timestep(c, w, batch, t, 0.f, temb, (char*)ws, hs(stream));
  g_no_events = false;
  return st;
}

dit_status dit_patch_embed(const dit_block_config* c, const dit_step_weights* w, int32_t batch, int32_t latent_dim,
                           const float* latent, void* x_img, void* workspace, size_t workspace_bytes,
                           dit_stream stream) {
  dit_status st = check_config(c);
  if (st || (st = check_step_weights(w))) return st;
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch < 0");
  if (latent_dim <= 0 || latent_dim % 64) return set_error(DIT_ERR_UNSUPPORTED, "latent_dim %d (multiple of 64)", latent_dim);
  if (batch == 0) return DIT_OK;
  if (!latent || !x_img || !aligned16(latent) || !aligned16(x_img))
    return set_error(DIT_ERR_INVALID_ARG, "latent/x_img NULL or not 16-byte aligned");
  if ((st = check_ws(workspace, workspace_bytes, patch_ws(c, batch, latent_dim)))) return st;
  return run_patch(c, w, batch, latent_dim, latent, x_img, (char*)workspace, hs(stream));
}

dit_status dit_final_layer(const dit_block_config* c, const dit_step_weights* w, int32_t batch, int32_t latent_dim,
                           const float* temb, const void* x_img, float* v, void* workspace, size_t workspace_bytes,
                           dit_stream stream) {
  dit_status st = check_config(c);
  if (st || (st = check_step_weights(w))) return st;
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch < 0");
  if (latent_dim <= 0 || latent_dim % 64) return set_error(DIT_ERR_UNSUPPORTED, "latent_dim %d (multiple of 64)", latent_dim);
  if (batch == 0) return DIT_OK;
  if (!temb || !x_img || !v || !aligned16(temb) || !aligned16(x_img) || !aligned16(v))
    return set_error(DIT_ERR_INVALID_ARG, "temb/x_img/v NULL or not 16-byte aligned");
  if ((st = check_ws(workspace, workspace_bytes, final_ws(c, batch)))) return st;
  return run_final(c, w, batch, latent_dim, temb, x_img, v, (char*)workspace, hs(stream));
}

size_t dit_denoise_workspace_bytes(const dit_block_config* c, int32_t batch, int32_t latent_dim) {
  if (check_config(c) != DIT_OK || batch < 0 || latent_dim <= 0) return 0;
  return step_layout(c, batch, latent_dim).total;
}

dit_status dit_denoise_step(const dit_block_config* c, const dit_step_weights* sw, const dit_block_weights* blocks,
                            int32_t n_blocks, int32_t batch, int32_t latent_dim, float t, float t_next,
                            float noise_level, float* latent, const void* x_txt, const float* noise, float* v_out,
                            void* workspace, size_t workspace_bytes, dit_stream stream) {
  dit_status st = check_config(c);
  if (st || (st = check_step_weights(sw))) return st;
  if (n_blocks < 0 || (n_blocks > 0 && !blocks)) return set_error(DIT_ERR_INVALID_ARG, "blocks NULL or n_blocks < 0");
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch < 0");
  if (latent_dim <= 0 || latent_dim % 64) return set_error(DIT_ERR_UNSUPPORTED, "latent_dim %d (multiple of 64)", latent_dim);
  float cx, cv, ce;
  if ((st = flow_coefficients(t, t_next, noise_level, noise != nullptr, &cx, &cv, &ce))) return st;
  if (batch == 0) return DIT_OK;
  if (!latent || !aligned16(latent) || (c->n_txt > 0 && (!x_txt || !aligned16(x_txt))) ||
      (v_out && !aligned16(v_out)))
    return set_error(DIT_ERR_INVALID_ARG, "latent/x_txt/v_out NULL or not 16-byte aligned");
  StepWs L = step_layout(c, batch, latent_dim);
  if ((st = check_ws(workspace, workspace_bytes, L.total))) return st;
  char* ws = (char*)workspace;
  float* temb = (float*)(ws + L.temb);
  void* ximg = ws + L.ximg;
  void* xtxt = ws + L.xtxt;
  float* v = v_out ? v_out : (float*)(ws + L.v);
  char* inner = ws + L.inner;
  for (int i = 0; i < n_blocks; i++)
    if ((st = check_block_args(c, &blocks[i], batch, temb, ximg, xtxt))) return st;
  hipStream_t s = hs(stream);
  const int B = batch, C = latent_dim;
  if ((st = run_timestep(c, sw, B, nullptr, t, temb, inner, s))) return st;
  if ((st = run_patch(c, sw, B, C, latent, ximg, inner, s))) return st;
  if (c->n_txt > 0)
    HIP_TRY(hipMemcpyAsync(xtxt, x_txt, (size_t)B * c->n_txt * c->hidden * esize(c->dtype), hipMemcpyDeviceToDevice, s));
  const BlockWs BL = block_layout(c, B);
  if (n_blocks > 0 && (st = check_ws(inner, workspace_bytes - L.inner, BL.total))) return st;
  if ((st = run_blocks(c, blocks, n_blocks, B, temb, ximg, xtxt, (float*)(ws + L.mods), inner, BL, false, s)))
    return st;
  if ((st = run_final(c, sw, B, C, temb, ximg, v, inner, s))) return st;
  TIMED("flow_step", 0, (noise_level > 0.f ? 16.0 : 12.0) * B * c->n_img * C, s,
        flow_update(latent, v, noise_level > 0.f ? noise : nullptr, (int64_t)B * c->n_img * C, cx, cv, ce, s));
  return DIT_OK;
}

// ---- TeaCache gate ----
namespace {
struct TeaCacheLayout {
  size_t hprev, resid, parts, sums, total;
};
TeaCacheLayout teacache_layout(const dit_block_config* c, int64_t B) {
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t n = (size_t)B * c->n_img * c->hidden;
  TeaCacheLayout L{};
  L.hprev = 0;
  L.resid = up(n * esize(c->dtype));
  L.parts = L.resid + up(n * 4);
  L.sums = L.parts + up(2 * sizeof(double) * TEACACHE_PARTS);
  L.total = L.sums + 256;
  return L;
}
}  // namespace

size_t dit_teacache_cache_bytes(const dit_block_config* c, int32_t batch) {
  if (check_config(c) != DIT_OK || batch < 0) return 0;
  return teacache_layout(c, batch).total;
}

dit_status dit_denoise_step_teacache(const dit_block_config* c, const dit_step_weights* sw,
                                     const dit_block_weights* blocks, int32_t n_blocks, int32_t batch,
                                     int32_t latent_dim, float t, float t_next, float noise_level, float* latent,
                                     const void* x_txt, const float* noise, float* v_out, dit_teacache_state* state,
                                     int32_t force, void* cache, size_t cache_bytes, int32_t* ran_blocks, double* rel,
                                     void* workspace, size_t workspace_bytes, dit_stream stream) {
  dit_status st = check_config(c);
  if (st || (st = check_step_weights(sw))) return st;
  if (n_blocks < 1 || !blocks) return set_error(DIT_ERR_INVALID_ARG, "the gated step needs n_blocks >= 1");
  if (!state) return set_error(DIT_ERR_INVALID_ARG, "state is NULL");
  if (batch < 0) return set_error(DIT_ERR_INVALID_ARG, "batch < 0");
  if (latent_dim <= 0 || latent_dim % 64) return set_error(DIT_ERR_UNSUPPORTED, "latent_dim %d (multiple of 64)", latent_dim);
  float cx, cv, ce;
  if ((st = flow_coefficients(t, t_next, noise_level, noise != nullptr, &cx, &cv, &ce))) return st;
  if (batch == 0) return DIT_OK;
  if (!latent || !aligned16(latent) || (c->n_txt > 0 && (!x_txt || !aligned16(x_txt))) ||
      (v_out && !aligned16(v_out)))
    return set_error(DIT_ERR_INVALID_ARG, "latent/x_txt/v_out NULL or not 16-byte aligned");
  const TeaCacheLayout TL = teacache_layout(c, batch);
  if (!cache || !aligned16(cache) || cache_bytes < TL.total)
    return set_error(DIT_ERR_WORKSPACE, "cache %zu bytes < %zu or not aligned", cache_bytes, TL.total);
  StepWs L = step_layout(c, batch, latent_dim);
  if ((st = check_ws(workspace, workspace_bytes, L.total))) return st;
  char* ws = (char*)workspace;
  float* temb = (float*)(ws + L.temb);
  void* ximg = ws + L.ximg;
  void* xtxt = ws + L.xtxt;
  float* v = v_out ? v_out : (float*)(ws + L.v);
  char* inner = ws + L.inner;
  for (int i = 0; i < n_blocks; i++)
    if ((st = check_block_args(c, &blocks[i], batch, temb, ximg, xtxt))) return st;
  hipStream_t s = hs(stream);
  const int B = batch, C = latent_dim, D = c->hidden;
  const int64_t n_act = (int64_t)B * c->n_img * D;
  char* cb = (char*)cache;
  float* resid = (float*)(cb + TL.resid);
  double* parts = (double*)(cb + TL.parts);
  double* sums = (double*)(cb + TL.sums);
  if ((st = run_timestep(c, sw, B, nullptr, t, temb, inner, s))) return st;
  if ((st = run_patch(c, sw, B, C, latent, ximg, inner, s))) return st;
  if (c->n_txt > 0)
    HIP_TRY(hipMemcpyAsync(xtxt, x_txt, (size_t)B * c->n_txt * D * esize(c->dtype), hipMemcpyDeviceToDevice, s));
  // block 0's modulated input: the first group's modulation GEMV and block 0's pre-attention LN
  // (both streams; the image rows are compared), in the block workspace the first block will overwrite
  const BlockWs BL = block_layout(c, B);
  if ((st = check_ws(inner, workspace_bytes - L.inner, BL.total))) return st;
  float* mods = (float*)(ws + L.mods);
  if ((st = run_modulation_group(c, blocks, std::min(n_blocks, MOD_GROUP), B, temb, mods, inner, BL, s))) return st;
  if ((st = run_ln(c, B, ximg, xtxt, mods, inner, BL, 0, D, s))) return st;
  const bool measure = state->has_prev != 0;
  TIMED("teacache_distance", 0, (measure ? 3.0 : 2.0) * n_act * esize(c->dtype), s,
        teacache_distance(inner + BL.h, cb + TL.hprev, B, c->n_img, c->n_txt, D, measure, parts, sums, c->dtype, s));
  double r = std::numeric_limits<double>::quiet_NaN();
  if (measure) {
    double hsums[2];
    HIP_TRY(hipMemcpyAsync(hsums, sums, sizeof hsums, hipMemcpyDeviceToHost, s));
    HIP_TRY(hipStreamSynchronize(s));
    r = hsums[1] > 0.0 ? hsums[0] / hsums[1] : (hsums[0] > 0.0 ? std::numeric_limits<double>::infinity() : 0.0);
  }
  int32_t run = 1;
  if (measure && !std::isfinite(r)) {
    run = 1;                 // a zero cached input: no meaningful distance, run the blocks
    state->accumulated = 0.0;
  } else if ((st = dit_teacache_gate(state, r, force, &run))) {
    return st;
  }
  state->has_prev = 1;
  if (run) {
    TIMED("small_elementwise", 0, 0, s, teacache_residual(ximg, resid, n_act, 0, c->dtype, s));
    if ((st = run_blocks(c, blocks, n_blocks, B, temb, ximg, xtxt, mods, inner, BL, true, s))) return st;
    TIMED("small_elementwise", 0, 0, s, teacache_residual(ximg, resid, n_act, 1, c->dtype, s));
    state->has_residual = 1;
  } else {
    TIMED("small_elementwise", 0, 0, s, teacache_residual(ximg, resid, n_act, 2, c->dtype, s));
  }
  if (ran_blocks) *ran_blocks = run;
  if (rel) *rel = r;
  if ((st = run_final(c, sw, B, C, temb, ximg, v, inner, s))) return st;
  TIMED("flow_step", 0, (noise_level > 0.f ? 16.0 : 12.0) * B * c->n_img * C, s,
        flow_update(latent, v, noise_level > 0.f ? noise : nullptr, (int64_t)B * c->n_img * C, cx, cv, ce, s));
  return DIT_OK;
}

dit_status dit_profile_begin(void) {
  std::lock_guard<std::mutex> g(g_prof.mu);
  for (auto& r : g_prof.recs) {
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  g_prof.recs.clear();
  g_prof.on.store(true, std::memory_order_release);
  return DIT_OK;
}

dit_status dit_profile_end(dit_kernel_stat* stats, int32_t capacity, int32_t* count) {
  std::lock_guard<std::mutex> g(g_prof.mu);
  g_prof.on.store(false, std::memory_order_release);
  std::map<std::string, dit_kernel_stat> agg;
  std::vector<std::string> order;
  dit_status st = DIT_OK;
  for (auto& r : g_prof.recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess && st == DIT_OK) st = set_error(DIT_ERR_HIP, "event timing failed: %s", hipGetErrorString(e));
    auto it = agg.find(r.name);
    if (it == agg.end()) {
      dit_kernel_stat k{};
      std::strncpy(k.name, r.name, sizeof(k.name) - 1);
      it = agg.emplace(r.name, k).first;
      order.push_back(r.name);
    }
    it->second.launches += 1;
    it->second.total_ms += ms;
    it->second.flops += r.flops;
    it->second.bytes += r.bytes;
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  g_prof.recs.clear();
  int32_t n = 0;
  for (auto& name : order) {
    if (stats && n < capacity) stats[n] = agg[name];
    n++;
  }
  if (count) *count = n;
  return st;
}

}  // extern "C"
