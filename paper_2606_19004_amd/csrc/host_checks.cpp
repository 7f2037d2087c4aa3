// Host-only half of the C ABI: the per-thread error text, argument checks that need no device
// (block configuration, flow-step coefficients) and the TeaCache gate. Plain C++ with no HIP
// dependency, so it also builds with g++ under the address and undefined-behaviour sanitizers.
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>

#include "host_checks.h"

namespace {
thread_local std::string g_err;
}

dit_status dit::set_error(dit_status s, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return s;
}

namespace dit {

dit_status check_config(const dit_block_config* c) {
  if (!c) return set_error(DIT_ERR_INVALID_ARG, "config is NULL");
  if (c->dtype != DIT_F32 && c->dtype != DIT_BF16) return set_error(DIT_ERR_INVALID_ARG, "dtype %d invalid", c->dtype);
  if (c->hidden <= 0 || c->heads <= 0 || c->head_dim <= 0 || c->mlp_hidden <= 0)
    return set_error(DIT_ERR_SHAPE, "hidden/heads/head_dim/mlp_hidden must be positive");
  if ((int64_t)c->hidden != (int64_t)c->heads * c->head_dim)
    return set_error(DIT_ERR_SHAPE, "hidden %d != heads %d * head_dim %d", c->hidden, c->heads, c->head_dim);
  if (c->head_dim != 64 && c->head_dim != 128) return set_error(DIT_ERR_UNSUPPORTED, "head_dim %d (64 or 128)", c->head_dim);
  if (c->hidden % 64 || c->mlp_hidden % 64) return set_error(DIT_ERR_UNSUPPORTED, "hidden and mlp_hidden must be multiples of 64");
  if (c->hidden > 4096) return set_error(DIT_ERR_UNSUPPORTED, "hidden %d > 4096", c->hidden);
  if (c->grid_h <= 0 || c->grid_w <= 0 || (int64_t)c->n_img != (int64_t)c->grid_h * c->grid_w)
    return set_error(DIT_ERR_SHAPE, "n_img %d != grid_h %d * grid_w %d", c->n_img, c->grid_h, c->grid_w);
  if (c->n_txt < 0) return set_error(DIT_ERR_SHAPE, "n_txt %d < 0", c->n_txt);
  // token counts enter 32-bit row arithmetic (B x S rows) downstream
  if ((int64_t)c->n_img + c->n_txt > (1 << 24))
    return set_error(DIT_ERR_UNSUPPORTED, "sequence of %lld tokens exceeds 2^24", (long long)c->n_img + c->n_txt);
  if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps)) return set_error(DIT_ERR_INVALID_ARG, "ln_eps must be positive");
  if (c->rope && (!(c->rope_theta > 0.f) || !std::isfinite(c->rope_theta)))
    return set_error(DIT_ERR_INVALID_ARG, "rope_theta must be positive");
  return DIT_OK;
}

dit_status flow_coefficients(float t, float t_next, float a, bool has_noise, float* cx, float* cv, float* ce) {
  if (!std::isfinite(t) || !std::isfinite(t_next) || !std::isfinite(a) || a < 0.f)
    return set_error(DIT_ERR_DOMAIN, "t, t_next and noise_level must be finite, noise_level >= 0");
  if (t_next > t) return set_error(DIT_ERR_DOMAIN, "t_next %g > t %g (the sampler runs from noise t=1 to data t=0)", t_next, t);
  double h = (double)t_next - (double)t;
  if (a == 0.f) {
    *cx = 1.f;
    *cv = (float)h;
    *ce = 0.f;
    return DIT_OK;
  }
  if (!(t > 0.f && t < 1.f)) return set_error(DIT_ERR_DOMAIN, "SDE step needs 0 < t < 1 (t = %g)", t);
  if (t_next < 0.f) return set_error(DIT_ERR_DOMAIN, "t_next %g < 0", t_next);
  if (!has_noise) return set_error(DIT_ERR_INVALID_ARG, "noise is NULL with noise_level > 0");
  double td = t, sigma = (double)a * std::sqrt(td / (1.0 - td));
  double k = sigma * sigma / (2.0 * td);
  // x + h (v + k (x + (1-t) v)) + sigma sqrt(-h) eps  =  (1 + h k) x + h (1 + k (1-t)) v + sigma sqrt(-h) eps
  *cx = (float)(1.0 + h * k);
  *cv = (float)(h * (1.0 + k * (1.0 - td)));
  *ce = (float)(sigma * std::sqrt(-h));
  return DIT_OK;
}

}  // namespace dit

using dit::set_error;

extern "C" {

int32_t dit_abi_version(void) { return DIT_ABI_VERSION; }

const char* dit_status_string(dit_status s) {
  switch (s) {
    case DIT_OK: return "ok";
    case DIT_ERR_INVALID_ARG: return "invalid argument";
    case DIT_ERR_SHAPE: return "inconsistent shape";
    case DIT_ERR_DOMAIN: return "argument outside the domain";
    case DIT_ERR_NAN: return "NaN or infinite input";
    case DIT_ERR_UNSUPPORTED: return "unsupported configuration";
    case DIT_ERR_HIP: return "HIP runtime error";
    case DIT_ERR_WORKSPACE: return "workspace missing, misaligned or too small";
  }
  return "unknown status";
}

const char* dit_last_error_message(void) { return g_err.c_str(); }

dit_status dit_teacache_init(dit_teacache_state* st, double threshold, const double* coef, int32_t n_coef) {
  if (!st) return set_error(DIT_ERR_INVALID_ARG, "state is NULL");
  if (!(threshold >= 0.0) || !std::isfinite(threshold)) return set_error(DIT_ERR_INVALID_ARG, "threshold %g < 0", threshold);
  if (n_coef < 0 || n_coef > 8 || (n_coef > 0 && !coef)) return set_error(DIT_ERR_INVALID_ARG, "n_coef %d (0..8)", n_coef);
  std::memset(st, 0, sizeof *st);
  st->threshold = threshold;
  st->n_coef = n_coef;
  for (int i = 0; i < n_coef; i++) {
    if (!std::isfinite(coef[i])) return set_error(DIT_ERR_INVALID_ARG, "coef[%d] not finite", i);
    st->coef[i] = coef[i];
  }
  return DIT_OK;
}

dit_status dit_teacache_gate(dit_teacache_state* st, double rel, int32_t force, int32_t* run_blocks) {
  if (!st || !run_blocks) return set_error(DIT_ERR_INVALID_ARG, "state / run_blocks is NULL");
  if (st->n_coef < 0 || st->n_coef > 8) return set_error(DIT_ERR_INVALID_ARG, "state n_coef %d (0..8)", st->n_coef);
  if (force || !st->has_prev || !st->has_residual) {
    st->accumulated = 0.0;
    *run_blocks = 1;
    return DIT_OK;
  }
  if (!std::isfinite(rel)) return set_error(DIT_ERR_NAN, "distance %g is not finite", rel);
  double v = rel;
  if (st->n_coef > 0) {   // Horner, highest power first
    v = 0.0;
    for (int i = 0; i < st->n_coef; i++) v = v * rel + st->coef[i];
  }
  st->accumulated += v;
  if (st->accumulated < st->threshold) {
    *run_blocks = 0;
  } else {
    st->accumulated = 0.0;
    *run_blocks = 1;
  }
  return DIT_OK;
}

}  // extern "C"
