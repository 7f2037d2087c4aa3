// Memory-bound and latency-bound kernels of the denoise step for gfx950:
//   flow_update    fused Euler / SDE latent update (fp32, 16-byte vector access)
//   flow_logprob   per-sample Gaussian log-density of an SDE step (fp64 sums)
//   ln_modulate    LayerNorm (fp32 statistics) + adaLN modulate, one wave per row
//   gemv           batched GEMV for the adaLN / timestep / final modulation vectors
//   reward_stats   per prompt-group mean, std, advantages, stable descending ranks
//   small helpers  SiLU, fp32->bf16 cast, timestep sinusoid, RoPE cos/sin table
#include "internal.h"

namespace dit {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------------------
// flow update: x' = cx*x + cv*v + ce*noise. The host folds the sampler step
// (Euler ODE or reverse-time SDE, both linear in x, v and noise) into these
// three coefficients in double precision.
// ---------------------------------------------------------------------------
template <bool NOISE>
__global__ void __launch_bounds__(256) flow_update_vec(float4* __restrict__ x, const float4* __restrict__ v,
                                                       const float4* __restrict__ e, int64_t n4,
                                                       float cx, float cv, float ce) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    float4 a = x[i], b = v[i];
    float4 r;
    r.x = fmaf(cx, a.x, cv * b.x);
    r.y = fmaf(cx, a.y, cv * b.y);
    r.z = fmaf(cx, a.z, cv * b.z);
    r.w = fmaf(cx, a.w, cv * b.w);
    if (NOISE) {
      float4 c = e[i];
      r.x = fmaf(ce, c.x, r.x);
      r.y = fmaf(ce, c.y, r.y);
      r.z = fmaf(ce, c.z, r.z);
      r.w = fmaf(ce, c.w, r.w);
    }
    x[i] = r;
  }
}

__global__ void flow_update_tail(float* x, const float* v, const float* e, int64_t start, int64_t n,
                                 float cx, float cv, float ce) {
  int64_t i = start + threadIdx.x;
  if (i < n) {
    float r = fmaf(cx, x[i], cv * v[i]);
    if (e) r = fmaf(ce, e[i], r);
    x[i] = r;
  }
}

__global__ void flow_update_scalar(float* x, const float* v, const float* e, int64_t n,
                                   float cx, float cv, float ce) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    float r = fmaf(cx, x[i], cv * v[i]);
    if (e) r = fmaf(ce, e[i], r);
    x[i] = r;
  }
}

// Log-density of an SDE step's output, one 1024-thread workgroup per sample: each thread sums
// (x_next - mean)^2 over a strided share of the sample in fp64 (the mean too is formed in fp64
// from the fp32 inputs), then the workgroup reduces in a fixed order.
template <bool VEC>
__global__ void __launch_bounds__(1024) flow_logprob_kernel(const float* __restrict__ x, const float* __restrict__ v,
                                                            const float* __restrict__ xn, int64_t n, double h,
                                                            double k1, double omt, double inv2var, double cst,
                                                            double* __restrict__ logp) {
  __shared__ double part[16];
  const int64_t base = (int64_t)blockIdx.x * n;
  double acc = 0.0;
  auto term = [&](float xf, float vf, float nf) {
    const double xd = xf, vd = vf;
    const double mean = xd + h * (vd + k1 * (xd + omt * vd));
    const double r = (double)nf - mean;
    acc = fma(r, r, acc);
  };
  if (VEC) {
    const float4* x4 = (const float4*)(x + base);
    const float4* v4 = (const float4*)(v + base);
    const float4* n4 = (const float4*)(xn + base);
    for (int64_t i = threadIdx.x; i < n / 4; i += 1024) {
      const float4 a = x4[i], b = v4[i], c = n4[i];
      term(a.x, b.x, c.x);
      term(a.y, b.y, c.y);
      term(a.z, b.z, c.z);
      term(a.w, b.w, c.w);
    }
  } else {
    for (int64_t i = threadIdx.x; i < n; i += 1024) term(x[base + i], v[base + i], xn[base + i]);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double s = 0.0;
    for (int w = 0; w < 16; w++) s += part[w];
    logp[blockIdx.x] = -s * inv2var + cst;
  }
}

hipError_t flow_logprob_launch(const float* x, const float* v, const float* xn, int batch, int64_t n, double h,
                               double k1, double omt, double inv2var, double cst, double* logp, hipStream_t s) {
  const bool vec = n % 4 == 0 && ((uintptr_t)x | (uintptr_t)v | (uintptr_t)xn) % 16 == 0;
  if (vec) flow_logprob_kernel<true><<<batch, 1024, 0, s>>>(x, v, xn, n, h, k1, omt, inv2var, cst, logp);
  else flow_logprob_kernel<false><<<batch, 1024, 0, s>>>(x, v, xn, n, h, k1, omt, inv2var, cst, logp);
  return hipGetLastError();
}

// TeaCache distance: each thread walks 8-element chunks of the image rows (grid-stride), sums
// |h - h_prev| and |h_prev| in fp64, and refreshes h_prev; one partial pair per workgroup.
template <typename T>
__global__ void __launch_bounds__(256) teacache_distance_kernel(const T* __restrict__ h, T* __restrict__ hp,
                                                                int64_t chunks, int64_t per_b, int n_txt, int S,
                                                                int D, int measure, double* __restrict__ part) {
  __shared__ double sd[4], sp[4];
  double ad = 0.0, ap = 0.0;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < chunks; q += (int64_t)gridDim.x * 256) {
    const int64_t e = q * 8, b = e / per_b, rem = e - b * per_b;
    const int64_t r = rem / D, c = rem - r * D;
    const T* src = h + (b * S + n_txt + r) * D + c;
    float a[8], p[8];
    load4<T>(src, a);
    load4<T>(src + 4, a + 4);
    if (measure) {
      load4<T>(hp + e, p);
      load4<T>(hp + e + 4, p + 4);
#pragma unroll
      for (int j = 0; j < 8; j++) {
        ad += fabs((double)a[j] - (double)p[j]);
        ap += fabs((double)p[j]);
      }
    }
    store4<T>(hp + e, a);
    store4<T>(hp + e + 4, a + 4);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    ad += __shfl_xor(ad, o, 64);
    ap += __shfl_xor(ap, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    sd[threadIdx.x >> 6] = ad;
    sp[threadIdx.x >> 6] = ap;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = sd[0] + sd[1] + sd[2] + sd[3];
    part[2 * blockIdx.x + 1] = sp[0] + sp[1] + sp[2] + sp[3];
  }
}

__global__ void teacache_sum_kernel(const double* __restrict__ part, int nparts, double* __restrict__ sums) {
  if (threadIdx.x == 0) {
    double a = 0.0, b = 0.0;
    for (int i = 0; i < nparts; i++) {
      a += part[2 * i];
      b += part[2 * i + 1];
    }
    sums[0] = a;
    sums[1] = b;
  }
}

hipError_t teacache_distance(const void* h, void* h_prev, int B, int n_img, int n_txt, int D, bool measure,
                             double* partials, double* sums, int dtype, hipStream_t s) {
  const int64_t per_b = (int64_t)n_img * D, chunks = B * per_b / 8;
  if (chunks == 0) return hipSuccess;
  const int grid = (int)std::min<int64_t>(TEACACHE_PARTS, cdiv(chunks, (int64_t)256));
  const int S = n_img + n_txt;
  if (dtype == DT_BF16)
    teacache_distance_kernel<u16><<<grid, 256, 0, s>>>((const u16*)h, (u16*)h_prev, chunks, per_b, n_txt, S, D,
                                                       measure, partials);
  else
    teacache_distance_kernel<float><<<grid, 256, 0, s>>>((const float*)h, (float*)h_prev, chunks, per_b, n_txt, S,
                                                         D, measure, partials);
  if (measure) teacache_sum_kernel<<<1, 64, 0, s>>>(partials, grid, sums);
  return hipGetLastError();
}

template <typename T, int MODE>
__global__ void __launch_bounds__(256) teacache_residual_kernel(T* __restrict__ x, float* __restrict__ r, int64_t n4) {
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < n4; q += (int64_t)gridDim.x * 256) {
    float a[4];
    load4<T>(x + 4 * q, a);
    float4 rv = MODE == 0 ? make_float4(0.f, 0.f, 0.f, 0.f) : *(const float4*)(r + 4 * q);
    if (MODE == 0) {
      *(float4*)(r + 4 * q) = make_float4(a[0], a[1], a[2], a[3]);
    } else if (MODE == 1) {
      *(float4*)(r + 4 * q) = make_float4(a[0] - rv.x, a[1] - rv.y, a[2] - rv.z, a[3] - rv.w);
    } else {
      float o[4] = {a[0] + rv.x, a[1] + rv.y, a[2] + rv.z, a[3] + rv.w};
      store4<T>(x + 4 * q, o);
    }
  }
}

hipError_t teacache_residual(void* x, float* r, int64_t n, int mode, int dtype, hipStream_t s) {
  const int64_t n4 = n / 4;
  if (n4 == 0) return hipSuccess;
  const int grid = (int)std::min<int64_t>(2048, cdiv(n4, (int64_t)256));
  if (dtype == DT_BF16) {
    if (mode == 0) teacache_residual_kernel<u16, 0><<<grid, 256, 0, s>>>((u16*)x, r, n4);
    else if (mode == 1) teacache_residual_kernel<u16, 1><<<grid, 256, 0, s>>>((u16*)x, r, n4);
    else teacache_residual_kernel<u16, 2><<<grid, 256, 0, s>>>((u16*)x, r, n4);
  } else {
    if (mode == 0) teacache_residual_kernel<float, 0><<<grid, 256, 0, s>>>((float*)x, r, n4);
    else if (mode == 1) teacache_residual_kernel<float, 1><<<grid, 256, 0, s>>>((float*)x, r, n4);
    else teacache_residual_kernel<float, 2><<<grid, 256, 0, s>>>((float*)x, r, n4);
  }
  return hipGetLastError();
}

hipError_t flow_update(float* x, const float* v, const float* noise, int64_t n, float cx, float cv, float ce,
                       hipStream_t s) {
  if (n <= 0) return hipSuccess;
  bool aligned = ((uintptr_t)x % 16 == 0) && ((uintptr_t)v % 16 == 0) && (!noise || (uintptr_t)noise % 16 == 0);
  if (aligned) {
    int64_t n4 = n / 4;
    if (n4 > 0) {
      int grid = (int)std::min<int64_t>(cdiv(n4, 256), 4096);
      if (noise)
        flow_update_vec<true><<<grid, 256, 0, s>>>((float4*)x, (const float4*)v, (const float4*)noise, n4, cx, cv, ce);
      else
        flow_update_vec<false><<<grid, 256, 0, s>>>((float4*)x, (const float4*)v, nullptr, n4, cx, cv, ce);
    }
    if (n % 4) flow_update_tail<<<1, 64, 0, s>>>(x, v, noise, n4 * 4, n, cx, cv, ce);
  } else {
    int grid = (int)std::min<int64_t>(cdiv(n, 256), 4096);
    flow_update_scalar<<<grid, 256, 0, s>>>(x, v, noise, n, cx, cv, ce);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// small helpers
// ---------------------------------------------------------------------------
__global__ void silu_kernel(const float* __restrict__ in, float* __restrict__ out, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) {
    float z = in[i];
    out[i] = z / (1.0f + __expf(-z));
  }
}
hipError_t silu_f32(const float* in, float* out, int64_t n, hipStream_t s) {
  if (n > 0) silu_kernel<<<cdiv(n, 256), 256, 0, s>>>(in, out, n);
  return hipGetLastError();
}

__global__ void cast_bf16_kernel(const float* __restrict__ in, u16* __restrict__ out, int64_t n) {
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) out[i] = from_f32<u16>(in[i]);
}
hipError_t cast_f32_to_bf16(const float* in, u16* out, int64_t n, hipStream_t s) {
  if (n > 0) cast_bf16_kernel<<<cdiv(n, 256), 256, 0, s>>>(in, out, n);
  return hipGetLastError();
}

// e[b] = [cos(1000 t f_j) ; sin(1000 t f_j)], f_j = 10000^(-j/128), evaluated in fp64.
__global__ void sinusoid_kernel(const float* t_dev, float t_scalar, float* e, int B) {
  int b = blockIdx.x, j = threadIdx.x;  // 128 threads
  double t = t_dev ? (double)t_dev[b] : (double)t_scalar;
  double f = exp(-log(10000.0) * (double)j / 128.0);
  double arg = 1000.0 * t * f;
  e[(int64_t)b * 256 + j] = (float)cos(arg);
  e[(int64_t)b * 256 + 128 + j] = (float)sin(arg);
}
hipError_t timestep_sinusoid(const float* t_dev, float t_scalar, float* e, int B, hipStream_t s) {
  if (B > 0) sinusoid_kernel<<<B, 128, 0, s>>>(t_dev, t_scalar, e, B);
  return hipGetLastError();
}

// tab[pos][i] = (cos, sin)(pos * theta^(-2i/m)), m = head_dim/2, i < m/2, in fp64.
__global__ void rope_table_kernel(float* tab, int npos, int head_dim, float theta) {
  int pairs = head_dim / 4;
  int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= npos * pairs) return;
  int pos = idx / pairs, i = idx % pairs;
  double m = head_dim / 2;
  double ang = (double)pos * pow((double)theta, -2.0 * i / m);
  tab[2 * idx] = (float)cos(ang);
  tab[2 * idx + 1] = (float)sin(ang);
}
hipError_t rope_table(float* tab, int npos, int head_dim, float theta, hipStream_t s) {
  int n = npos * (head_dim / 4);
  if (n > 0) rope_table_kernel<<<cdiv(n, 256), 256, 0, s>>>(tab, npos, head_dim, theta);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// LayerNorm + modulate. One 64-lane wave per row; each lane owns CH chunks of
// 8 consecutive elements (16-byte bf16 or 32-byte fp32 accesses), so a row of
// D <= 512*CH stays in registers for the two-pass mean / variance.
// ---------------------------------------------------------------------------
template <typename T> struct Vec8;
template <> struct Vec8<u16> {
  static __device__ __forceinline__ void load(const u16* p, float* f) {
    uint4 u = *(const uint4*)p;
    uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  static __device__ __forceinline__ void store(u16* p, const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; i++)
      w[i] = (uint32_t)from_f32<u16>(f[2 * i]) | ((uint32_t)from_f32<u16>(f[2 * i + 1]) << 16);
    *(uint4*)p = make_uint4(w[0], w[1], w[2], w[3]);
  }
};
template <> struct Vec8<float> {
  static __device__ __forceinline__ void load(const float* p, float* f) {
    float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w; f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  static __device__ __forceinline__ void store(float* p, const float* f) {
    *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
    *(float4*)(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
  }
};

template <typename T, int CH>
__global__ void __launch_bounds__(256) ln_modulate_kernel(LnArgs a) {
  int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  int lane = threadIdx.x & 63;
  int64_t total = a.rows[0] + a.rows[1];
  if (row >= total) return;
  int s = row < a.rows[0] ? 0 : 1;
  int64_t m = s == 0 ? row : row - a.rows[0];
  int64_t b = m / a.xmap[s].rows_per_batch;
  const T* x = (const T*)a.x[s] + row_offset(a.xmap[s], m);
  T* out = (T*)a.out + row_offset(a.omap[s], m);
  const float* shift = a.mod[s] + b * a.mod_bstride + a.shift_off;
  const float* scale = a.mod[s] + b * a.mod_bstride + a.scale_off;
  const int D = a.D;

  float v[CH][8];
  float sum = 0.f;
#pragma unroll
  for (int c = 0; c < CH; c++) {
    int k = (c * 64 + lane) * 8;
    if (k < D) {
      Vec8<T>::load(x + k, v[c]);
#pragma unroll
      for (int i = 0; i < 8; i++) sum += v[c][i];
    } else {
#pragma unroll
      for (int i = 0; i < 8; i++) v[c][i] = 0.f;
    }
  }
  float mean = wave_sum(sum) / (float)D;
  float sq = 0.f;
#pragma unroll
  for (int c = 0; c < CH; c++) {
    int k = (c * 64 + lane) * 8;
    if (k < D) {
#pragma unroll
      for (int i = 0; i < 8; i++) {
        float d = v[c][i] - mean;
        sq += d * d;
      }
    }
  }
  float rstd = rsqrtf(wave_sum(sq) / (float)D + a.eps);
#pragma unroll
  for (int c = 0; c < CH; c++) {
    int k = (c * 64 + lane) * 8;
    if (k < D) {
      float4 sh0 = *(const float4*)(shift + k), sh1 = *(const float4*)(shift + k + 4);
      float4 sc0 = *(const float4*)(scale + k), sc1 = *(const float4*)(scale + k + 4);
      float sh[8] = {sh0.x, sh0.y, sh0.z, sh0.w, sh1.x, sh1.y, sh1.z, sh1.w};
      float sc[8] = {sc0.x, sc0.y, sc0.z, sc0.w, sc1.x, sc1.y, sc1.z, sc1.w};
      float o[8];
#pragma unroll
      for (int i = 0; i < 8; i++) o[i] = fmaf((v[c][i] - mean) * rstd, 1.0f + sc[i], sh[i]);
      Vec8<T>::store(out + k, o);
    }
  }
}

template <typename T>
static hipError_t ln_launch(const LnArgs& a, hipStream_t s) {
  int64_t total = a.rows[0] + a.rows[1];
  if (total == 0) return hipSuccess;
  int grid = cdiv(total, 4);
  int ch = cdiv(a.D, 512);
  if (ch <= 1) ln_modulate_kernel<T, 1><<<grid, 256, 0, s>>>(a);
  else if (ch <= 2) ln_modulate_kernel<T, 2><<<grid, 256, 0, s>>>(a);
  else if (ch <= 4) ln_modulate_kernel<T, 4><<<grid, 256, 0, s>>>(a);
  else if (ch <= 6) ln_modulate_kernel<T, 6><<<grid, 256, 0, s>>>(a);
  else ln_modulate_kernel<T, 8><<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}
hipError_t ln_modulate(const LnArgs& a, int dtype, hipStream_t s) {
  return dtype == DT_BF16 ? ln_launch<u16>(a, s) : ln_launch<float>(a, s);
}

// ---------------------------------------------------------------------------
// batched GEMV: out[s][b][n] = W[s][n][:] . in[b][:] + bias[s][n], B <= 16 per
// pass. A wave owns 4 weight rows and streams them once (16-byte loads), with
// the fp32 input read through L1/L2; lanes split K and reduce at the end.
// ---------------------------------------------------------------------------
template <typename T, int BMAX>
__global__ void __launch_bounds__(256) gemv_kernel(GemvArgs a, int b0, int nb) {
  constexpr int R = 4;
  int s = blockIdx.y;
  int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int n0 = (blockIdx.x * 4 + wave) * R;
  if (n0 >= a.N) return;
  const T* W = (const T*)a.W[s];
  float acc[R][BMAX];
#pragma unroll
  for (int r = 0; r < R; r++)
#pragma unroll
    for (int b = 0; b < BMAX; b++) acc[r][b] = 0.f;
  for (int k = lane * 8; k < a.K; k += 512) {
    float w[R][8];
#pragma unroll
    for (int r = 0; r < R; r++) {
      if (n0 + r < a.N) Vec8<T>::load(W + (int64_t)(n0 + r) * a.K + k, w[r]);
      else
#pragma unroll
        for (int i = 0; i < 8; i++) w[r][i] = 0.f;
    }
#pragma unroll
    for (int b = 0; b < BMAX; b++) {
      if (b < nb) {
        float x[8];
        Vec8<float>::load(a.in + (int64_t)(b0 + b) * a.in_bstride + k, x);
#pragma unroll
        for (int r = 0; r < R; r++)
#pragma unroll
          for (int i = 0; i < 8; i++) acc[r][b] = fmaf(w[r][i], x[i], acc[r][b]);
      }
    }
  }
  const T* bias = (const T*)a.bias[s];
#pragma unroll
  for (int r = 0; r < R; r++) {
#pragma unroll
    for (int b = 0; b < BMAX; b++) {
      float v = wave_sum(acc[r][b]);
      if (lane == 0 && b < nb && n0 + r < a.N) {
        if (bias) v += to_f32(bias[n0 + r]);
        a.out[s][(int64_t)(b0 + b) * a.out_bstride + n0 + r] = v;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// bf16 weights: an MFMA skinny GEMM. The fp32 input (at most 16 samples per
// pass) is split once into bf16 hi + lo parts (x = hi + lo to ~2^-16), laid out
// [2][16][K]; each wave then streams 32 weight rows once and multiplies them
// against both parts with v_mfma_f32_16x16x32_bf16 (samples are the MFMA's
// 16-wide N dimension), so HBM bandwidth, not VALU FMAs, sets the time.
// A workgroup owns 32 weight rows and splits K over its 4 waves.
// ---------------------------------------------------------------------------
__global__ void split_hilo_kernel(const float* __restrict__ in, int64_t stride, int b0, int nb, int K, int silu,
                                  u16* __restrict__ out) {
  int k = blockIdx.x * 256 + threadIdx.x, b = blockIdx.y;
  if (k >= K) return;
  float x = 0.f;
  if (b < nb) {
    x = in[(int64_t)(b0 + b) * stride + k];
    if (silu) x = x / (1.0f + __expf(-x));
  }
  __bf16 hi = (__bf16)x;
  __bf16 lo = (__bf16)(x - (float)hi);
  out[(int64_t)b * K + k] = __builtin_bit_cast(u16, hi);
  out[(int64_t)(16 + b) * K + k] = __builtin_bit_cast(u16, lo);
}

// One workgroup = 16 RB weight rows (RB row blocks of 16, each the A operand of its own MFMA
// chain); its 4 waves take every 4th 32-deep k step and the partial sums meet in LDS, so each
// row block streams with 4 independent load chains. Every k step of a wave reads the split input
// (2 x 1 KB from L2) once for its RB row blocks (RB x 1 KB of weights), so more row blocks per
// workgroup mean fewer re-reads of the input per weight byte: with the weights cold in HBM, RB = 8
// (one k step per wave in flight, 180 registers) streams the 1.81 GB of a step's modulation
// weights in 426 us against 467 us for RB = 4 with two k steps in flight. Small GEMVs (the
// timestep and final-layer ones, a few MB of weights) are bound by the latency of each wave's chain
// of k steps instead: they take fewer rows per workgroup (more workgroups) and, with DEPTH > 0, keep
// DEPTH of a wave's k steps in flight (the loads of step i + DEPTH - 1 are issued before the MFMAs
// of step i; loads past the wave's last step are clamped to that step, so that every load is
// unconditional and the compiler can count the loads in flight). The sums run in the same order
// either way.
template <int RB, int U, int DEPTH = 0>
__global__ void __launch_bounds__(256) gemv_mfma_kernel(GemvArgs a, const u16* __restrict__ xs, int b0, int nb) {
  __shared__ f32x4 part[4][RB][64];
  const int s = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int n0 = blockIdx.x * 16 * RB;
  const int K = a.K, nks = K / 32;
  const int r16 = lane & 15, kq = (lane >> 4) * 8;
  // operand A: rows n0 + 16 j + r16 (clamped; results of clamped rows are dropped)
  const u16* W = (const u16*)a.W[s];
  const u16* w[RB];
#pragma unroll
  for (int j = 0; j < RB; j++) w[j] = W + (int64_t)min(n0 + 16 * j + r16, a.N - 1) * K + kq;
  // operand B: sample r16, hi and lo parts
  const u16* xh = xs + (int64_t)r16 * K + kq;
  const u16* xl = xs + (int64_t)(16 + r16) * K + kq;
  f32x4 acc[RB];
#pragma unroll
  for (int j = 0; j < RB; j++) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  if constexpr (DEPTH == 0) {
    int ks = wave;
    for (; ks + 4 * (U - 1) < nks; ks += 4 * U) {
      bf16x8 fw[U][RB], fh[U], fl[U];
#pragma unroll
      for (int u = 0; u < U; u++) {
        int k = 32 * (ks + 4 * u);
#pragma unroll
        for (int j = 0; j < RB; j++) fw[u][j] = *(const bf16x8*)(w[j] + k);
        fh[u] = *(const bf16x8*)(xh + k);
        fl[u] = *(const bf16x8*)(xl + k);
      }
#pragma unroll
      for (int u = 0; u < U; u++)
#pragma unroll
        for (int j = 0; j < RB; j++) {
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[u][j], fh[u], acc[j], 0, 0, 0);
          acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[u][j], fl[u], acc[j], 0, 0, 0);
        }
    }
    for (; ks < nks; ks += 4) {
      int k = 32 * ks;
      bf16x8 fh = *(const bf16x8*)(xh + k), fl = *(const bf16x8*)(xl + k);
#pragma unroll
      for (int j = 0; j < RB; j++) {
        bf16x8 fw = *(const bf16x8*)(w[j] + k);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw, fh, acc[j], 0, 0, 0);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw, fl, acc[j], 0, 0, 0);
      }
    }
  } else {
    // this wave's k steps are wave + 4 i, i < nloc; the first nmain of them run pipelined
    const int nloc = nks > wave ? (nks - wave + 3) / 4 : 0;
    const int nmain = nloc - nloc % DEPTH;
    bf16x8 fw[DEPTH][RB], fh[DEPTH], fl[DEPTH];
    auto load = [&](int i, int slot) {
      const int k = 32 * (wave + 4 * i);
#pragma unroll
      for (int j = 0; j < RB; j++) fw[slot][j] = *(const bf16x8*)(w[j] + k);
      fh[slot] = *(const bf16x8*)(xh + k);
      fl[slot] = *(const bf16x8*)(xl + k);
    };
    auto mma = [&](int slot) {
#pragma unroll
      for (int j = 0; j < RB; j++) {
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[slot][j], fh[slot], acc[j], 0, 0, 0);
        acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fw[slot][j], fl[slot], acc[j], 0, 0, 0);
      }
    };
    if (nmain > 0) {
#pragma unroll
      for (int d = 0; d < DEPTH - 1; d++) load(d, d);
      __builtin_amdgcn_sched_barrier(0);
      for (int i = 0; i < nmain; i += DEPTH) {
#pragma unroll
        for (int u = 0; u < DEPTH; u++) {
          load(min(i + u + DEPTH - 1, nloc - 1), (u + DEPTH - 1) % DEPTH);
          __builtin_amdgcn_sched_barrier(0);   // keep the loads ahead of this step's MFMAs
          mma(u);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
    }
    for (int i = nmain; i < nloc; i++) {
      load(i, 0);
      mma(0);
    }
  }
#pragma unroll
  for (int j = 0; j < RB; j++) part[wave][j][lane] = acc[j];
  __syncthreads();
  if (wave != 0) return;
  // sum the 4 partials in a fixed order (deterministic)
#pragma unroll
  for (int q = 1; q < 4; q++)
#pragma unroll
    for (int j = 0; j < RB; j++) {
      f32x4 p = part[q][j][lane];
#pragma unroll
      for (int r = 0; r < 4; r++) acc[j][r] += p[r];
    }
  // accumulator register r of lane l in block j: weight row 16 j + 4 (l / 16) + r, sample l % 16
  const int b = lane & 15;
  if (b >= nb) return;
  const u16* bias = (const u16*)a.bias[s];
  float* out = a.out[s] + (int64_t)(b0 + b) * a.out_bstride;
#pragma unroll
  for (int j = 0; j < RB; j++)
#pragma unroll
    for (int r = 0; r < 4; r++) {
      int n = n0 + 16 * j + 4 * (lane >> 4) + r;
      if (n < a.N) out[n] = acc[j][r] + (bias ? to_f32(bias[n]) : 0.f);
    }
}

hipError_t gemv_bf16(const GemvArgs& a, u16* xs, int silu_in, hipStream_t s) {
  if (a.N == 0 || a.B == 0) return hipSuccess;
  for (int b0 = 0; b0 < a.B; b0 += 16) {
    int nb = std::min(16, a.B - b0);
    split_hilo_kernel<<<dim3(cdiv(a.K, 256), 16), 256, 0, s>>>(a.in, a.in_bstride, b0, nb, a.K, silu_in, xs);
    // rows per workgroup by grid size: the step's batched modulation (1.8 GB of weights) streams
    // best with 128; a single block's (0.2 GB) with 64; the timestep and final-layer GEMVs (a few
    // MB) need more workgroups and a pipelined k chain (lab, same box: 30 -> 18 us for 3072 x 3072,
    // 31 -> 20 us for 6144 x 3072, bit-identical)
    const int64_t ns = a.nstreams;
    if ((int64_t)cdiv(a.N, 128) * ns >= 1024)
      gemv_mfma_kernel<8, 1><<<dim3(cdiv(a.N, 128), a.nstreams), 256, 0, s>>>(a, xs, b0, nb);
    else if ((int64_t)cdiv(a.N, 64) * ns >= 256)
      gemv_mfma_kernel<4, 2><<<dim3(cdiv(a.N, 64), a.nstreams), 256, 0, s>>>(a, xs, b0, nb);
    else if ((int64_t)cdiv(a.N, 32) * ns >= 192)
      gemv_mfma_kernel<2, 1, 2><<<dim3(cdiv(a.N, 32), a.nstreams), 256, 0, s>>>(a, xs, b0, nb);
    else
      gemv_mfma_kernel<1, 1, 4><<<dim3(cdiv(a.N, 16), a.nstreams), 256, 0, s>>>(a, xs, b0, nb);
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t gemv_launch(const GemvArgs& a, hipStream_t s) {
  dim3 grid(cdiv(a.N, 16), a.nstreams);
  for (int b0 = 0; b0 < a.B; b0 += 16) {
    int nb = std::min(16, a.B - b0);
    if (nb <= 4) gemv_kernel<T, 4><<<grid, 256, 0, s>>>(a, b0, nb);
    else if (nb <= 8) gemv_kernel<T, 8><<<grid, 256, 0, s>>>(a, b0, nb);
    else gemv_kernel<T, 16><<<grid, 256, 0, s>>>(a, b0, nb);
  }
  return hipGetLastError();
}
hipError_t gemv(const GemvArgs& a, int dtype, hipStream_t s) {
  if (a.N == 0 || a.B == 0) return hipSuccess;
  return dtype == DT_BF16 ? gemv_launch<u16>(a, s) : gemv_launch<float>(a, s);
}

// ---------------------------------------------------------------------------
// per-group reward statistics. One 256-thread workgroup per group; rewards of
// the group in LDS; fp64 sums; rank of seed i = #{j : r_j > r_i or
// (r_j == r_i and j < i)}, so order[rank_i] = i is the stable descending sort
// (ties by index), computed without atomics and bit-exactly.
// ---------------------------------------------------------------------------
__device__ double block_sum_f64(double v, double* red) {
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// status[0] = 0 when every one of the `count` rewards is finite, else the non-finite code; one
// workgroup strides over the input (the reward matrix is small: groups x seeds)
__global__ void __launch_bounds__(256) reward_check_kernel(const float* __restrict__ rw, int64_t count,
                                                           int32_t bad_code, int32_t* status) {
  __shared__ int any[4];
  int bad = 0;
  for (int64_t i = threadIdx.x; i < count; i += 256) bad |= !isfinite(rw[i]);
  bad = __any(bad);
  if ((threadIdx.x & 63) == 0) any[threadIdx.x >> 6] = bad;
  __syncthreads();
  if (threadIdx.x == 0) status[0] = (any[0] | any[1] | any[2] | any[3]) ? bad_code : 0;
}

__global__ void __launch_bounds__(256) reward_stats_kernel(const float* __restrict__ rw, int n, float adv_eps,
                                                           int k, float* mean, float* stdv, float* adv,
                                                           int32_t* order, int32_t* sel, const int32_t* status) {
  extern __shared__ float sr[];               // n rewards, then n ints of order
  __shared__ double red[4];
  if (status && status[0] != 0) return;       // non-finite input: nothing is written
  int32_t* so = (int32_t*)(sr + n);
  int g = blockIdx.x;
  const float* r = rw + (int64_t)g * n;
  double part = 0.0;
  for (int i = threadIdx.x; i < n; i += 256) {
    float x = r[i];
    sr[i] = x;
    part += (double)x;
  }
  double mu = block_sum_f64(part, red) / (double)n;   // block_sum syncs after the LDS fill
  part = 0.0;
  for (int i = threadIdx.x; i < n; i += 256) {
    double d = (double)sr[i] - mu;
    part += d * d;
  }
  double sd = sqrt(block_sum_f64(part, red) / (double)n);
  if (threadIdx.x == 0) {
    if (mean) mean[g] = (float)mu;
    if (stdv) stdv[g] = (float)sd;
  }
  for (int i = threadIdx.x; i < n; i += 256) {
    float ri = sr[i];
    if (adv) adv[(int64_t)g * n + i] = sd > 0.0 ? (float)(((double)ri - mu) / (sd + (double)adv_eps)) : 0.0f;
    int rank = 0;
    for (int j = 0; j < n; j++) {
      float rj = sr[j];
      rank += (rj > ri) || (rj == ri && j < i);
    }
    so[rank] = i;
  }
  __syncthreads();
  int top = (k + 1) / 2;
  for (int i = threadIdx.x; i < n; i += 256)
    if (order) order[(int64_t)g * n + i] = so[i];
  for (int q = threadIdx.x; q < k; q += 256)
    if (sel) sel[(int64_t)g * k + q] = so[q < top ? q : n - k + q];
}

hipError_t reward_stats(const float* r, int G, int n, float adv_eps, int k, float* mean, float* stdv,
                        float* adv, int32_t* order, int32_t* sel, int32_t* status, int32_t bad_code, hipStream_t s) {
  if (G == 0) return hipSuccess;
  if (status) {
    reward_check_kernel<<<1, 256, 0, s>>>(r, (int64_t)G * n, bad_code, status);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  size_t lds = (size_t)n * 8;
  reward_stats_kernel<<<G, 256, lds, s>>>(r, n, adv_eps, k, mean, stdv, adv, order, sel, status);
  return hipGetLastError();
}

}  // namespace dit
