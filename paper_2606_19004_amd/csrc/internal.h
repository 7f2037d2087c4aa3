// Internal interfaces between the C ABI layer (api.hip) and the gfx950 kernels.
// Nothing here crosses the library boundary.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace dit {

typedef unsigned short u16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// ---------------------------------------------------------------------------
// element access: bf16 storage (as u16 bits) or fp32, math always in fp32
// ---------------------------------------------------------------------------
__device__ __forceinline__ float to_f32(float x) { return x; }
__device__ __forceinline__ float to_f32(u16 x) { return __uint_as_float(((uint32_t)x) << 16); }
template <typename T> __device__ __forceinline__ T from_f32(float x);
template <> __device__ __forceinline__ float from_f32<float>(float x) { return x; }
template <> __device__ __forceinline__ u16 from_f32<u16>(float x) {
  return __builtin_bit_cast(u16, (__bf16)x);  // round to nearest even (v_cvt_pk_bf16_f32)
}

// four consecutive elements as fp32 (16-byte aligned for fp32, 8-byte for bf16), and back
template <typename T> __device__ __forceinline__ void load4(const T* p, float* f);
template <> __device__ __forceinline__ void load4<u16>(const u16* p, float* f) {
  uint2 u = *(const uint2*)p;
  f[0] = __uint_as_float(u.x << 16);
  f[1] = __uint_as_float(u.x & 0xffff0000u);
  f[2] = __uint_as_float(u.y << 16);
  f[3] = __uint_as_float(u.y & 0xffff0000u);
}
template <> __device__ __forceinline__ void load4<float>(const float* p, float* f) {
  float4 a = *(const float4*)p;
  f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
}
// two fp32 values as packed bf16 (a in the low half), one v_cvt_pk_bf16_f32 (round to nearest even)
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}
template <typename T> __device__ __forceinline__ void store4(T* p, const float* f);
template <> __device__ __forceinline__ void store4<u16>(u16* p, const float* f) {
  *(uint2*)p = make_uint2(pack_bf16x2(f[0], f[1]), pack_bf16x2(f[2], f[3]));
}
template <> __device__ __forceinline__ void store4<float>(float* p, const float* f) {
  *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
}

// ---------------------------------------------------------------------------
// row addressing: logical row m of a [rows][cols] operand lives at element
//   (m / rows_per_batch) * batch_stride + (m % rows_per_batch) * row_stride + offset
// which lets one stream's tokens be a strided slice of a joint [B][S][...] buffer.
// ---------------------------------------------------------------------------
struct RowMap {
  int64_t rows_per_batch;
  int64_t batch_stride;
  int64_t row_stride;
  int64_t offset;
};
__host__ __device__ __forceinline__ int64_t row_offset(const RowMap& r, int64_t m) {
  int64_t b = m / r.rows_per_batch;
  return b * r.batch_stride + (m - b * r.rows_per_batch) * r.row_stride + r.offset;
}
inline RowMap contiguous_rows(int64_t cols) { return RowMap{1, cols, 0, 0}; }

__host__ __device__ __forceinline__ int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// ---------------------------------------------------------------------------
// GEMM: C[m][n] = epilogue( sum_k A[m][k] W[n][k] + bias[n] ), W stored [N][K]
// ---------------------------------------------------------------------------
enum Epi { EPI_STORE = 0, EPI_GELU = 1, EPI_RESID = 2, EPI_QKV = 3 };

struct GemmProblem {
  const void* A;  RowMap amap;   // rows of A (K contiguous)
  const void* W;                 // [N][K] contiguous
  const void* bias;              // [N] (weight dtype) or null
  void* C;        RowMap cmap;   // output rows (N contiguous)
  int M, N, K;
  // EPI_RESID: C = C + gate[b][n] * y with b = m / cmap.rows_per_batch
  const float* gate; int64_t gate_bstride;
  // EPI_QKV: 2D RoPE on columns [0, 2*hidden) (q and k) of image rows
  const float* rope_tab;         // [npos][head_dim/4] pairs (cos, sin), null = no RoPE
  int grid_w, head_dim, hidden, rope_npos;
};

struct GemmPair {              // up to two problems (image stream, text stream) in one launch
  GemmProblem p[2];
  int nprob;
};

enum Dtype { DT_F32 = 0, DT_BF16 = 1 };

hipError_t gemm(const GemmPair& pr, int epi, int dtype, bool out_f32, hipStream_t s);

// ---------------------------------------------------------------------------
// attention
// ---------------------------------------------------------------------------
struct AttnArgs {
  const void* q; const void* k; const void* v; void* o;
  int B, H, S, d;
  int64_t qs_b, qs_s, qs_h;
  int64_t os_b, os_s, os_h;
  float scale;
};
hipError_t attention(const AttnArgs& a, int dtype, hipStream_t s);

// ---------------------------------------------------------------------------
// memory-bound kernels
// ---------------------------------------------------------------------------
// LayerNorm (no affine) + modulate over the rows of up to two streams.
// out = LN(x)(1 + scale[b]) + shift[b]; shift at mod[s] + b*mod_bstride + shift_off.
struct LnArgs {
  const void* x[2]; RowMap xmap[2];
  void* out;        RowMap omap[2];
  const float* mod[2]; int64_t mod_bstride; int shift_off, scale_off;
  int64_t rows[2];     // rows per stream (B * N_s)
  int D; float eps;
};
hipError_t ln_modulate(const LnArgs& a, int dtype, hipStream_t s);

// out[s][b][n] = sum_k W[s][n][k] in[b][k] + bias[s][n]  (fp32 in/out, W in weight dtype)
// up to GEMV_SLOTS independent weight matrices (same N, K, input) in one launch: the two streams of a
// block, or the modulation of several blocks at once
constexpr int GEMV_SLOTS = 16;
struct GemvArgs {
  const void* W[GEMV_SLOTS]; const void* bias[GEMV_SLOTS]; float* out[GEMV_SLOTS];
  int64_t out_bstride;
  const float* in; int64_t in_bstride;
  int N, K, B, nstreams;
};
hipError_t gemv(const GemvArgs& a, int dtype, hipStream_t s);   // VALU (fp32 weights)
// bf16 weights through MFMA; xs = scratch [2][16][K] bf16; silu_in applies SiLU to the input first;
// K must be a multiple of 32
hipError_t gemv_bf16(const GemvArgs& a, u16* xs, int silu_in, hipStream_t s);

hipError_t silu_f32(const float* in, float* out, int64_t n, hipStream_t s);
hipError_t cast_f32_to_bf16(const float* in, u16* out, int64_t n, hipStream_t s);
hipError_t timestep_sinusoid(const float* t_dev, float t_scalar, float* e, int B, hipStream_t s);
hipError_t rope_table(float* tab, int npos, int head_dim, float theta, hipStream_t s);
// per-sample Gaussian log-density of an SDE step: logp[b] = -sum (xn - mean)^2 * inv2var + cst,
// mean = x + h (v + k1 (x + omt v))
hipError_t flow_logprob_launch(const float* x, const float* v, const float* xn, int batch, int64_t n, double h,
                               double k1, double omt, double inv2var, double cst, double* logp, hipStream_t s);
// TeaCache: per-block partial sums of |h - h_prev| and |h_prev| over the image rows of the joint
// buffer h ([B][S][D], image rows at offset n_txt) against h_prev ([B][N_i][D]), summed in a fixed
// order into sums[2] (skipped when !measure); h_prev is then overwritten with h.
hipError_t teacache_distance(const void* h, void* h_prev, int B, int n_img, int n_txt, int D, bool measure,
                             double* partials, double* sums, int dtype, hipStream_t s);
// residual r (fp32) of the activation x (n elements): mode 0 r = x, 1 r = x - r, 2 x = x + r
hipError_t teacache_residual(void* x, float* r, int64_t n, int mode, int dtype, hipStream_t s);
constexpr int TEACACHE_PARTS = 512;
hipError_t flow_update(float* x, const float* v, const float* noise, int64_t n,
                       float cx, float cv, float ce, hipStream_t s);
// status (device, nullable): a check pass first writes 0 or bad_code (any reward non-finite) there,
// and the statistics kernel writes nothing when it is non-zero
hipError_t reward_stats(const float* r, int G, int n, float adv_eps, int k,
                        float* mean, float* stdv, float* adv, int32_t* order, int32_t* sel,
                        int32_t* status, int32_t bad_code, hipStream_t s);

}  // namespace dit
