// GEMMs of the MMDiT block on gfx950: C = epilogue(A W^T + bias), W stored [N][K].
//
// bf16 path: LDS-staged MFMA kernel (v_mfma_f32_32x32x16_bf16, fp32 accumulate).
//   * Computed as C^T = W A^T: MFMA operand "A" = 32 rows of W, operand "B" =
//     32 rows of A; both are K-contiguous, so every lane reads one 16-byte
//     chunk per fragment (ds_read_b128). The accumulator gives each lane one
//     token row m and runs of 4 consecutive output features n, which is what
//     the epilogues need (RoPE pairs (2i, 2i+1) sit in one lane).
//   * Tiles of A and W move HBM -> LDS with buffer_load ... lds (no VGPR
//     staging), double-buffered. Out-of-range rows use an offset past the
//     buffer's num_records, which the hardware turns into zeros.
//   * LDS rows are 64 bf16 = 8 chunks of 16 bytes; chunk c of row r is stored
//     at chunk slot c ^ (r % 8), so the 8 lanes of a ds_read_b128 phase hit 8
//     different bank groups.
//   * Workgroups are dispatched round-robin over the 8 XCDs; tile t is given
//     to workgroup ids so that each XCD owns one contiguous range of tiles,
//     ordered in groups of 8 M-tiles so concurrently running tiles share A and
//     W panels in that XCD's L2.
// fp32 path: VALU tiles (64x64, 4x4 per thread) with the same epilogue.
#include "internal.h"

namespace dit {

// ---------------------------------------------------------------------------
// epilogue on 4 consecutive output features n..n+3 of row m
// ---------------------------------------------------------------------------
__device__ __forceinline__ float gelu_tanh_f(float z) {
  // 0.5 z (1 + tanh(u)) = z * sigmoid(2u), u = sqrt(2/pi) (z + 0.044715 z^3)
  float u2 = 2.0f * 0.7978845608028654f * fmaf(0.044715f * z, z * z, z);
  return z / (1.0f + __builtin_amdgcn_exp2f(-u2 * 1.4426950408889634f));
}

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
template <typename T> __device__ __forceinline__ void store4(T* p, const float* f);
template <> __device__ __forceinline__ void store4<u16>(u16* p, const float* f) {
  uint2 u;
  u.x = (uint32_t)from_f32<u16>(f[0]) | ((uint32_t)from_f32<u16>(f[1]) << 16);
  u.y = (uint32_t)from_f32<u16>(f[2]) | ((uint32_t)from_f32<u16>(f[3]) << 16);
  *(uint2*)p = u;
}
template <> __device__ __forceinline__ void store4<float>(float* p, const float* f) {
  *(float4*)p = make_float4(f[0], f[1], f[2], f[3]);
}

template <int EPI, typename TW, typename TC>
__device__ __forceinline__ void epilogue4(const GemmProblem& P, int m, int n, float* v) {
  if (P.bias) {
    float b[4];
    load4<TW>((const TW*)P.bias + n, b);
#pragma unroll
    for (int q = 0; q < 4; q++) v[q] += b[q];
  }
  if (EPI == EPI_GELU) {
#pragma unroll
    for (int q = 0; q < 4; q++) v[q] = gelu_tanh_f(v[q]);
  }
  TC* out = (TC*)P.C + row_offset(P.cmap, m) + n;
  if (EPI == EPI_RESID) {
    int64_t b = m / P.cmap.rows_per_batch;
    float4 g = *(const float4*)(P.gate + b * P.gate_bstride + n);
    float x[4];
    load4<TC>(out, x);
    v[0] = fmaf(g.x, v[0], x[0]);
    v[1] = fmaf(g.y, v[1], x[1]);
    v[2] = fmaf(g.z, v[2], x[2]);
    v[3] = fmaf(g.w, v[3], x[3]);
  }
  if (EPI == EPI_QKV) {
    if (P.rope_tab && n < 2 * P.hidden) {
      // image token i = m % rows_per_batch at grid (i / grid_w, i % grid_w);
      // head dims [0, d/2) rotate by the row, [d/2, d) by the column
      int i = (int)(m % P.cmap.rows_per_batch);
      int dd = n % P.head_dim;
      int half = P.head_dim >> 1;
      int pos = dd < half ? i / P.grid_w : i % P.grid_w;
      int pr = (dd % half) >> 1;   // pair index of (dd, dd+1)
      const float* cs = P.rope_tab + ((int64_t)pos * (P.head_dim >> 2) + pr) * 2;
      float4 t = *(const float4*)cs;   // pairs pr and pr+1
      float a0 = v[0], b0 = v[1], a1 = v[2], b1 = v[3];
      v[0] = a0 * t.x - b0 * t.y;
      v[1] = a0 * t.y + b0 * t.x;
      v[2] = a1 * t.z - b1 * t.w;
      v[3] = a1 * t.w + b1 * t.z;
    }
  }
  store4<TC>(out, v);
}

// ---------------------------------------------------------------------------
// bf16 MFMA GEMM
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void* lds_ptr_t;

__device__ __forceinline__ void tile_coords(int tl, int mt, int nt, int& tm, int& tn) {
  constexpr int GROUP_M = 8;
  int per_group = GROUP_M * nt;
  int group = tl / per_group;
  int first_m = group * GROUP_M;
  int gm = min(mt - first_m, GROUP_M);
  int in_group = tl - group * per_group;
  tm = first_m + in_group % gm;
  tn = in_group / gm;
}

template <int BM, int BN, int WM, int WN, int EPI, bool OUTF32>
__global__ void __launch_bounds__(256) gemm_bf16_kernel(GemmPair pr, int tiles0, int total_tiles) {
  constexpr int BK = 64;
  constexpr int WTM = BM / WM, WTN = BN / WN;  // wave tile (m, n)
  constexpr int TJ = WTM / 32, TI = WTN / 32;  // 32x32 MFMA blocks per wave along m and n
  constexpr int A_LOADS = BM / 32, W_LOADS = BN / 32;  // 8-row groups loaded per wave per k-tile
  constexpr int A_BYTES = BM * BK * 2, W_BYTES = BN * BK * 2;
  static_assert(WM * WN == 4, "four waves");
#if defined(__HIP_DEVICE_COMPILE__)  // the buffer-resource builtins exist only in the device pass
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  // XCD-aware tile index
  int per = gridDim.x >> 3;
  int t = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (t >= total_tiles) return;
  int pi = t < tiles0 ? 0 : 1;
  const GemmProblem& P = pr.p[pi];
  int tl = pi == 0 ? t : t - tiles0;
  int mt = cdiv(P.M, BM), nt = cdiv(P.N, BN);
  int tm, tn;
  tile_coords(tl, mt, nt, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int K = P.K;

  // buffer resources; rows outside the matrix get an offset beyond num_records -> zeros
  const uint32_t OOB = 0x80000000u;
  __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc((void*)P.A, (short)0, 0x7fffffff, 0x00020000);
  __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc((void*)P.W, (short)0, 0x7fffffff, 0x00020000);
  const int lrow = lane >> 3;                    // row inside an 8-row group
  const int lchunk = (lane & 7) ^ lrow;          // global chunk this lane fetches (slot = lane & 7)
  uint32_t aoff[A_LOADS], woff[W_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; i++) {
    int m = m0 + (wave * A_LOADS + i) * 8 + lrow;
    aoff[i] = m < P.M ? (uint32_t)(row_offset(P.amap, m) * 2 + lchunk * 16) : OOB;
  }
#pragma unroll
  for (int i = 0; i < W_LOADS; i++) {
    int n = n0 + (wave * W_LOADS + i) * 8 + lrow;
    woff[i] = n < P.N ? (uint32_t)((int64_t)n * K * 2 + lchunk * 16) : OOB;
  }

  auto issue = [&](int kt, int buf) {
    char* sa = smem + buf * (A_BYTES + W_BYTES);
    char* sw = sa + A_BYTES;
    int soff = kt * BK * 2;
#pragma unroll
    for (int i = 0; i < A_LOADS; i++)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (lds_ptr_t)(sa + (wave * A_LOADS + i) * 1024), 16, aoff[i], soff, 0, 0);
#pragma unroll
    for (int i = 0; i < W_LOADS; i++)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(sw + (wave * W_LOADS + i) * 1024), 16, woff[i], soff, 0, 0);
  };

  f32x16 acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; i++)
#pragma unroll
    for (int j = 0; j < TJ; j++)
#pragma unroll
      for (int r = 0; r < 16; r++) acc[i][j][r] = 0.f;

  const int wm = wave / WN, wn = wave % WN;
  const int half = lane >> 5, l32 = lane & 31, sw8 = lane & 7;
  const int nk = K / BK;
  issue(0, 0);
  for (int kt = 0; kt < nk; kt++) {
    __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of tile kt have landed in LDS
    __syncthreads();                 // ... and everyone's; the other buffer is free again
    if (kt + 1 < nk) issue(kt + 1, (kt + 1) & 1);
    const char* sa = smem + (kt & 1) * (A_BYTES + W_BYTES);
    const char* sw = sa + A_BYTES;
#pragma unroll
    for (int s = 0; s < BK / 16; s++) {
      const int slot = ((2 * s + half) ^ sw8) * 16;
      bf16x8 fw[TI], fa[TJ];
#pragma unroll
      for (int i = 0; i < TI; i++) fw[i] = *(const bf16x8*)(sw + (wn * WTN + 32 * i + l32) * 128 + slot);
#pragma unroll
      for (int j = 0; j < TJ; j++) fa[j] = *(const bf16x8*)(sa + (wm * WTM + 32 * j + l32) * 128 + slot);
#pragma unroll
      for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[i], fa[j], acc[i][j], 0, 0, 0);
    }
  }

  // accumulator (i, j), register r: n = 32i + 8(r/4) + 4*half + r%4, m = 32j + lane%32
#pragma unroll
  for (int i = 0; i < TI; i++) {
#pragma unroll
    for (int j = 0; j < TJ; j++) {
      int m = m0 + wm * WTM + 32 * j + l32;
      if (m >= P.M) continue;
#pragma unroll
      for (int g = 0; g < 4; g++) {
        int n = n0 + wn * WTN + 32 * i + 8 * g + 4 * half;
        if (n < P.N) {
          float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
          if (OUTF32) epilogue4<EPI, u16, float>(P, m, n, v);
          else epilogue4<EPI, u16, u16>(P, m, n, v);
        }
      }
    }
  }
#endif
}

template <int BM, int BN, int WM, int WN, int EPI, bool OUTF32>
static hipError_t launch_bf16(const GemmPair& pr, hipStream_t s) {
  int tiles[2] = {0, 0};
  for (int i = 0; i < pr.nprob; i++)
    if (pr.p[i].M > 0 && pr.p[i].N > 0) tiles[i] = cdiv(pr.p[i].M, BM) * cdiv(pr.p[i].N, BN);
  int total = tiles[0] + tiles[1];
  if (total == 0) return hipSuccess;
  size_t lds = 2 * (size_t)(BM + BN) * 64 * 2;
  static bool attr_set[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  if (lds > 65536 && dev < 64 && !attr_set[dev]) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_kernel<BM, BN, WM, WN, EPI, OUTF32>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set[dev] = true;
  }
  int grid = 8 * cdiv(total, 8);
  gemm_bf16_kernel<BM, BN, WM, WN, EPI, OUTF32><<<grid, 256, lds, s>>>(pr, tiles[0], total);
  return hipGetLastError();
}

template <int EPI, bool OUTF32>
static hipError_t dispatch_bf16(const GemmPair& pr, hipStream_t s) {
  int maxn = 0;
  int64_t big_tiles = 0;
  for (int i = 0; i < pr.nprob; i++) {
    maxn = std::max(maxn, pr.p[i].N);
    big_tiles += (int64_t)cdiv(pr.p[i].M, 256) * cdiv(pr.p[i].N, 256);
  }
  if (maxn <= 64) return launch_bf16<64, 64, 2, 2, EPI, OUTF32>(pr, s);
  if (big_tiles < 512) return launch_bf16<128, 128, 2, 2, EPI, OUTF32>(pr, s);
  return launch_bf16<256, 256, 2, 2, EPI, OUTF32>(pr, s);
}

// ---------------------------------------------------------------------------
// fp32 VALU GEMM (64x64 tile, 16-deep k slices, 4x4 outputs per thread)
// ---------------------------------------------------------------------------
template <int EPI>
__global__ void __launch_bounds__(256) gemm_f32_kernel(GemmPair pr, int tiles0, int total_tiles) {
  constexpr int BM = 64, BN = 64, BK = 16;
  __shared__ float sa[BK][BM + 4];
  __shared__ float sw[BK][BN + 4];
  int t = blockIdx.x;
  if (t >= total_tiles) return;
  int pi = t < tiles0 ? 0 : 1;
  const GemmProblem& P = pr.p[pi];
  int tl = pi == 0 ? t : t - tiles0;
  int nt = cdiv(P.N, BN);
  int m0 = (tl / nt) * BM, n0 = (tl % nt) * BN;
  const float* A = (const float*)P.A;
  const float* W = (const float*)P.W;
  int tid = threadIdx.x;
  int tr = tid / 16, tc = tid % 16;   // 16 x 16 threads, each 4 rows x 4 consecutive n
  float acc[4][4] = {};
  // loader: 64 rows x 16 k per operand = 1024 values, 4 per thread
  int lr = tid / 4, lk = (tid % 4) * 4;
  int64_t arow = m0 + lr < P.M ? row_offset(P.amap, m0 + lr) : -1;
  int64_t wrow = n0 + lr < P.N ? (int64_t)(n0 + lr) * P.K : -1;
  for (int k0 = 0; k0 < P.K; k0 += BK) {
#pragma unroll
    for (int q = 0; q < 4; q++) {
      int k = k0 + lk + q;
      sa[lk + q][lr] = (arow >= 0 && k < P.K) ? A[arow + k] : 0.f;
      sw[lk + q][lr] = (wrow >= 0 && k < P.K) ? W[wrow + k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < BK; k++) {
      float a[4], w[4];
#pragma unroll
      for (int q = 0; q < 4; q++) a[q] = sa[k][tr * 4 + q];
#pragma unroll
      for (int q = 0; q < 4; q++) w[q] = sw[k][tc * 4 + q];
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; i++) {
    int m = m0 + tr * 4 + i, n = n0 + tc * 4;
    if (m < P.M && n < P.N) epilogue4<EPI, float, float>(P, m, n, acc[i]);
  }
}

template <int EPI>
static hipError_t launch_f32(const GemmPair& pr, hipStream_t s) {
  int tiles[2] = {0, 0};
  for (int i = 0; i < pr.nprob; i++)
    if (pr.p[i].M > 0 && pr.p[i].N > 0) tiles[i] = cdiv(pr.p[i].M, 64) * cdiv(pr.p[i].N, 64);
  int total = tiles[0] + tiles[1];
  if (total == 0) return hipSuccess;
  gemm_f32_kernel<EPI><<<total, 256, 0, s>>>(pr, tiles[0], total);
  return hipGetLastError();
}

hipError_t gemm(const GemmPair& pr, int epi, int dtype, bool out_f32, hipStream_t s) {
  if (dtype == DT_F32) {
    switch (epi) {
      case EPI_STORE: return launch_f32<EPI_STORE>(pr, s);
      case EPI_GELU: return launch_f32<EPI_GELU>(pr, s);
      case EPI_RESID: return launch_f32<EPI_RESID>(pr, s);
      case EPI_QKV: return launch_f32<EPI_QKV>(pr, s);
    }
    return hipErrorInvalidValue;
  }
  if (out_f32) {
    if (epi == EPI_STORE) return dispatch_bf16<EPI_STORE, true>(pr, s);
    return hipErrorInvalidValue;
  }
  switch (epi) {
    case EPI_STORE: return dispatch_bf16<EPI_STORE, false>(pr, s);
    case EPI_GELU: return dispatch_bf16<EPI_GELU, false>(pr, s);
    case EPI_RESID: return dispatch_bf16<EPI_RESID, false>(pr, s);
    case EPI_QKV: return dispatch_bf16<EPI_QKV, false>(pr, s);
  }
  return hipErrorInvalidValue;
}

}  // namespace dit
