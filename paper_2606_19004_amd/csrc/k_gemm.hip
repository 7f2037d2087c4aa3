// GEMMs of the MMDiT block on gfx950: C = epilogue(A W^T + bias), W stored [N][K].
//
// bf16 path: LDS-staged MFMA kernel with fp32 accumulation.
//   * Computed as C^T = W A^T: MFMA operand "A" = rows of W, operand "B" = rows
//     of A; both are K-contiguous, so every lane reads one 16-byte chunk per
//     fragment (ds_read_b128). The accumulator gives each lane one token row m
//     and runs of 4 consecutive output features n, which is what the epilogues
//     need (RoPE pairs (2i, 2i+1) sit in one lane).
//   * Tiles of A and W move HBM -> LDS with buffer_load ... lds (no VGPR
//     staging). Out-of-range rows use an offset past the buffer's num_records,
//     which the hardware turns into zeros. In the large tile a wave's refill of
//     one operand is a single burst of up to four such loads under one M0 value
//     (the instruction offset steps the LDS destination by 1 KB): a load issued
//     between MFMAs holds the wave's issue for ~17 cycles, and the M0 save and
//     restore around each load for ~13 more, while back-to-back loads share it.
//   * LDS rows are 64 bf16 = 8 chunks of 16 bytes; chunk c of row r is stored
//     at slot c ^ ((r >> 1) & 7), so every lane group that a ds_read_b128 of a
//     fragment is served in hits 16 different bank groups of the 64-bank LDS.
//   * The large tile (256 x 256 x 64, v_mfma_f32_16x16x32_bf16) runs 8 waves
//     (2 per SIMD), each 64 rows x 128 features, and keeps three LDS stages of
//     A and two of W (160 KB), so the activation rows are requested two k-tiles
//     before use. Fragments of the next 32-deep k step load while the current
//     step's MFMAs run; the k-tile barrier sits at the last step, whose
//     fragments are already in registers. The refill is split between the two
//     steps of a k-tile (W after the barrier, A in the other step), and each
//     wave lowers its issue priority as it advances between barriers, so the
//     two waves of a SIMD share the matrix pipe instead of one running ahead
//     and idling at the barrier. Smaller problems use 128 x 128 or 64 x 64
//     tiles with v_mfma_f32_32x32x16_bf16 and two stages of each.
//   * Epilogue: bias, gate vectors and the RoPE table are staged in LDS per
//     tile; the gated residual reads of a wave's whole sub-tile are issued at
//     once.
//   * Workgroups are dispatched round-robin over the 8 XCDs; tile t is given
//     to workgroup ids so that each XCD owns one contiguous range of tiles,
//     ordered in groups of 8 M-tiles so concurrently running tiles share A and
//     W panels in that XCD's L2.
// fp32 path: VALU tiles (64x64, 4x4 per thread) with the same epilogue.
#include <atomic>
#include <type_traits>

#include "internal.h"

namespace dit {

// ---------------------------------------------------------------------------
// epilogue on 4 consecutive output features n..n+3 of row m
// ---------------------------------------------------------------------------
__device__ __forceinline__ float gelu_tanh_f(float z) {
  // 0.5 z (1 + tanh(u)) = z * sigmoid(2u), u = sqrt(2/pi) (z + 0.044715 z^3), and
  // sigmoid(2u) = 1 / (1 + 2^(-2u log2 e)) with -2u log2 e = z (K1 + K2 z^2)
  constexpr float K1 = -2.0f * 0.7978845608028654f * 1.4426950408889634f;
  constexpr float K2 = K1 * 0.044715f;
  return z * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z * fmaf(K2, z * z, K1)));
}


// Per-row epilogue state, computed once per output row m.
struct RowEpi {
  int64_t off;   // element offset of row m in C
  int64_t gate;  // element offset of the row's gate vector (EPI_RESID)
  int rpos, cpos;  // grid row / column of an image token (EPI_QKV with RoPE)
};

__device__ __forceinline__ RowEpi row_epi(const GemmProblem& P, int m) {
  RowEpi r;
  int rpb = (int)P.cmap.rows_per_batch;
  int b = m / rpb, i = m - b * rpb;
  r.off = (int64_t)b * P.cmap.batch_stride + (int64_t)i * P.cmap.row_stride + P.cmap.offset;
  r.gate = (int64_t)b * P.gate_bstride;
  r.rpos = P.grid_w > 0 ? i / P.grid_w : 0;
  r.cpos = P.grid_w > 0 ? i - r.rpos * P.grid_w : 0;
  return r;
}

template <int EPI, typename TW, typename TC>
__device__ __forceinline__ void epilogue4(const GemmProblem& P, const RowEpi& R, int n, float* v) {
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
  TC* out = (TC*)P.C + R.off + n;
  if (EPI == EPI_RESID) {
    float4 g = *(const float4*)(P.gate + R.gate + n);
    float x[4];
    load4<TC>(out, x);
    v[0] = fmaf(g.x, v[0], x[0]);
    v[1] = fmaf(g.y, v[1], x[1]);
    v[2] = fmaf(g.z, v[2], x[2]);
    v[3] = fmaf(g.w, v[3], x[3]);
  }
  if (EPI == EPI_QKV) {
    if (P.rope_tab && n < 2 * P.hidden) {
      // head dims [0, d/2) rotate by the token's grid row, [d/2, d) by its column;
      // n..n+3 hold the pairs (pr, pr+1) of one half (head_dim is a power of two)
      int dd = n & (P.head_dim - 1);
      int hh = P.head_dim >> 1;
      int pos = dd < hh ? R.rpos : R.cpos;
      int pr = (dd & (hh - 1)) >> 1;
      float4 t = *(const float4*)(P.rope_tab + ((int64_t)pos * (P.head_dim >> 2) + pr) * 2);
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
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// Direct-to-LDS 16-byte-per-lane buffer load (M0 = LDS destination of lane 0), written as inline
// assembly so that the compiler does not track it: with LDS addresses chosen at run time it cannot
// prove that a later LDS read does not alias the load, and would wait for all loads in flight. The
// caller's explicit s_waitcnt vmcnt is the only synchronisation for these loads. M0 is reserved by
// the compiler, so the sequence saves it in a scratch SGPR and restores it after issuing the load
// (the destination is taken from M0 when the load issues). rsrc is a raw buffer descriptor (base,
// stride 0, num_records, flags).
__device__ __forceinline__ void dma_b128(u32x4_t rsrc, uint32_t m0v, uint32_t voff, uint32_t soff) {
  uint32_t saved;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\tbuffer_load_dwordx4 %2, %3, %4 offen lds\n\t"
               "s_mov_b32 m0, %0"
               : "=&s"(saved) : "s"(m0v), "v"(voff), "s"(rsrc), "s"(soff) : "memory");
}

// N (3 or 4) direct-to-LDS loads sharing one M0: destination M0 + 1024 i + 16 lane, global offset
// v[i] + 1024 i (the instruction offset moves both addresses)
template <int N>
__device__ __forceinline__ void dma_burst(u32x4_t rsrc, uint32_t m0v, const uint32_t* v, uint32_t soff) {
  uint32_t saved;
  if constexpr (N == 4)
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                 "buffer_load_dwordx4 %2, %6, %7 offen lds\n\t"
                 "buffer_load_dwordx4 %3, %6, %7 offen offset:1024 lds\n\t"
                 "buffer_load_dwordx4 %4, %6, %7 offen offset:2048 lds\n\t"
                 "buffer_load_dwordx4 %5, %6, %7 offen offset:3072 lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(saved) : "s"(m0v), "v"(v[0]), "v"(v[1]), "v"(v[2]), "v"(v[3]), "s"(rsrc), "s"(soff) : "memory");
  else
    asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
                 "buffer_load_dwordx4 %2, %5, %6 offen lds\n\t"
                 "buffer_load_dwordx4 %3, %5, %6 offen offset:1024 lds\n\t"
                 "buffer_load_dwordx4 %4, %5, %6 offen offset:2048 lds\n\t"
                 "s_mov_b32 m0, %0"
                 : "=&s"(saved) : "s"(m0v), "v"(v[0]), "v"(v[1]), "v"(v[2]), "s"(rsrc), "s"(soff) : "memory");
}

// Exchange lanes 16-31 of x with lanes 0-15 of y and lanes 48-63 of x with lanes 32-47 of y.
__device__ __forceinline__ void swap16(uint32_t& x, uint32_t& y) {
  const auto r = __builtin_amdgcn_permlane16_swap(x, y, false, false);
  x = r[0];
  y = r[1];
}

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

// LDS swizzle key of tile row r (rows of 128 bytes = 64 bf16 of k): chunk c of row r lives in
// 16-byte slot c ^ f(r). Measured service rule of ds_read_b128 on this chip: the 64 lanes are
// served as four groups of 16, a group being the lanes that agree in lane bit 5 and in the
// parity of lane bits 2..4; a group takes as many cycles as the largest number of its lanes
// that hit one 16-byte bank group ((address / 16) mod 16) at different addresses. With
// f(r) = (r / 2) mod 8 every group of a 16x16x32 or a 32x32x16 fragment read hits 16 distinct
// bank groups, so a wave's read takes the minimum four cycles.
__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Instructions of one kind placed after MFMA q when n of them are spread evenly over the first
// `span` MFMAs of a k step.
__host__ __device__ constexpr int spread(int q, int n, int span) {
  return span <= 0 ? (q == 0 ? n : 0) : ((q + 1 < span ? q + 1 : span) * n) / span - ((q < span ? q : span) * n) / span;
}

// Scheduling hints for one k step of NM MFMAs: NV direct-to-LDS loads spread over the first half
// of the MFMAs, ND fragment reads over the first three quarters.
template <int NM, int NV, int ND, int Q = 0>
__device__ __forceinline__ void sched_step() {
  if constexpr (Q < NM) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA
    constexpr int v = spread(Q, NV, NM / 2), d = spread(Q, ND, 3 * NM / 4);
    if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);   // VMEM loads
    if constexpr (d > 0) __builtin_amdgcn_sched_group_barrier(0x100, d, 0);   // LDS reads
    sched_step<NM, NV, ND, Q + 1>();
  }
}

// One MFMA on MS x MS blocks: v_mfma_f32_32x32x16_bf16 (MS = 32) or v_mfma_f32_16x16x32_bf16
// (MS = 16). Both take one 8-element bf16 fragment per lane for each operand.
template <int MS> struct Mfma;
template <> struct Mfma<32> {
  typedef f32x16 acc_t;
  static constexpr int KS = 16;   // k depth of one instruction
  static __device__ __forceinline__ acc_t run(bf16x8 a, bf16x8 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mfma<16> {
  typedef f32x4 acc_t;
  static constexpr int KS = 32;
  static __device__ __forceinline__ acc_t run(bf16x8 a, bf16x8 b, acc_t c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};

// MS = MFMA block size (32 or 16); under sustained load with random operands the 16x16x32
// form delivers more MFMA throughput per watt on this chip.
// TRI (256 x 256 tiles only): three LDS stages for A and two for W (160 KB), so the activation
// operand is loaded two k-tiles ahead.
template <int BM, int BN, int WM, int WN, int EPI, bool OUTF32, int MS = 32, bool TRI = false>
__global__ void __launch_bounds__(WM * WN * 64) gemm_bf16_kernel(GemmPair pr, int tiles0, int total_tiles) {
  typedef typename Mfma<MS>::acc_t acc_t;
  constexpr int NACC = sizeof(acc_t) / 4;              // accumulator registers per block
  constexpr int KS = Mfma<MS>::KS;
  constexpr int NW = WM * WN;
  constexpr int BK = 64;
  constexpr int WTM = BM / WM, WTN = BN / WN;          // wave tile (m, n)
  constexpr int TJ = WTM / MS, TI = WTN / MS;          // MFMA blocks per wave along m and n
  constexpr int A_LOADS = BM / 8 / NW, W_LOADS = BN / 8 / NW;  // 8-row groups each wave loads per k-tile
  constexpr int A_BYTES = BM * BK * 2, W_BYTES = BN * BK * 2;
  static_assert(A_LOADS >= 1 && W_LOADS >= 1, "every wave loads at least one row group");
  static_assert(!TRI || (BM == 256 && (BN == 256 || BN == 192)), "three A stages only for 256-row tiles");
#if defined(__HIP_DEVICE_COMPILE__)  // the buffer-resource builtins exist only in the device pass
  extern __shared__ __attribute__((aligned(1024))) char smem[];

  // XCD-aware tile index
  int per = gridDim.x >> 3;
  int t = (blockIdx.x & 7) * per + (blockIdx.x >> 3);
  if (t >= total_tiles) return;
  int pi = t < tiles0 ? 0 : 1;
  const GemmProblem P = pr.p[pi];   // a copy: its fields stay in registers instead of being reloaded per use
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
  // a wave-load writes 8 rows x 8 slots (lane -> row lane/8, slot lane%8) and fetches chunk slot ^ f(row)
  const int lrow = lane >> 3;
  uint32_t aoff[A_LOADS], woff[W_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; i++) {
    int g = wave * A_LOADS + i;
    int chunk = (lane & 7) ^ swz(8 * g + lrow);
    int m = m0 + 8 * g + lrow;
    aoff[i] = m < P.M ? (uint32_t)(row_offset(P.amap, m) * 2 + chunk * 16) : OOB;
  }
#pragma unroll
  for (int i = 0; i < W_LOADS; i++) {
    int g = wave * W_LOADS + i;
    int chunk = (lane & 7) ^ swz(8 * g + lrow);
    int n = n0 + 8 * g + lrow;
    woff[i] = n < P.N ? (uint32_t)((int64_t)n * K * 2 + chunk * 16) : OOB;
  }
  // TRI layout: [W0][W1][A0][A1][A2]; tile kt uses W stage kt % 2 and A stage kt % 3
  auto stage_w = [&](int kt) -> char* { return smem + (kt & 1) * W_BYTES; };
  auto stage_a = [&](int kt) -> char* { return smem + 2 * W_BYTES + (kt % 3) * A_BYTES; };
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  const uint64_t pa64 = (uint64_t)P.A, pw64 = (uint64_t)P.W;
  // refills as one burst per operand: offsets carry -1024 i plus a 4 KB bias taken back from the base
  constexpr bool BA = TRI && (A_LOADS == 3 || A_LOADS == 4), BW = TRI && (W_LOADS == 3 || W_LOADS == 4);
  const uint64_t pa64b = pa64 - (BA ? 4096u : 0u), pw64b = pw64 - (BW ? 4096u : 0u);
  // (with the bias every in-range offset stays below 2^31 + 4 KB, the records bound; rows outside the
  // matrix move to 3 GiB, past it, and still read zeros)
  const u32x4_t ra4 = {(uint32_t)pa64b, (uint32_t)(pa64b >> 32) & 0xffffu, BA ? 0x80001000u : 0x7fffffffu, 0x00020000u};
  const u32x4_t rw4 = {(uint32_t)pw64b, (uint32_t)(pw64b >> 32) & 0xffffu, BW ? 0x80001000u : 0x7fffffffu, 0x00020000u};
  uint32_t aoffb[A_LOADS], woffb[W_LOADS];
#pragma unroll
  for (int i = 0; i < A_LOADS; i++) aoffb[i] = BA ? (aoff[i] == OOB ? 0xC0000000u : aoff[i]) + 4096u - 1024u * i : aoff[i];
#pragma unroll
  for (int i = 0; i < W_LOADS; i++) woffb[i] = BW ? (woff[i] == OOB ? 0xC0000000u : woff[i]) + 4096u - 1024u * i : woff[i];
  const uint32_t smem_lds = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
  auto issue_a = [&](int kt) {
    const uint32_t sa = smem_lds + (uint32_t)(stage_a(kt) - smem);
    const uint32_t soff = kt * BK * 2;
#pragma unroll
    for (int i = 0; i < (BA ? 0 : A_LOADS); i++) dma_b128(ra4, sa + (wave_s * A_LOADS + i) * 1024, aoffb[i], soff);
    if constexpr (BA) dma_burst<A_LOADS>(ra4, sa + wave_s * A_LOADS * 1024, aoffb, soff);
  };
  auto issue_w = [&](int kt) {
    const uint32_t sw = smem_lds + (uint32_t)(stage_w(kt) - smem);
    const uint32_t soff = kt * BK * 2;
#pragma unroll
    for (int i = 0; i < (BW ? 0 : W_LOADS); i++) dma_b128(rw4, sw + (wave_s * W_LOADS + i) * 1024, woffb[i], soff);
    if constexpr (BW) dma_burst<W_LOADS>(rw4, sw + wave_s * W_LOADS * 1024, woffb, soff);
  };
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

  acc_t acc[TI][TJ];
#pragma unroll
  for (int i = 0; i < TI; i++)
#pragma unroll
    for (int j = 0; j < TJ; j++)
#pragma unroll
      for (int r = 0; r < NACC; r++) acc[i][j][r] = 0.f;

  const int wm = wave / WN, wn = wave % WN;
  // lane -> (fragment row inside an MS-row block, 8-element k chunk inside a KS step)
  const int frow = lane % MS, lkc = lane / MS;
  const int nk = K / BK;
  int fwk[TI], fak[TJ];
#pragma unroll
  for (int i = 0; i < TI; i++) fwk[i] = swz(wn * WTN + MS * i + frow);
#pragma unroll
  for (int j = 0; j < TJ; j++) fak[j] = swz(wm * WTM + MS * j + frow);
  const int wrow0 = (wn * WTN + frow) * 128, arow0 = (wm * WTM + frow) * 128;
  // fragments of k step s, register-double-buffered so step s+1 loads while step s multiplies
  bf16x8 fw[2][TI], fa[2][TJ];
  auto frags = [&](int buf, int s, int rb) {   // TRI: buf is the k-tile index
    const char* sa = TRI ? stage_a(buf) : smem + buf * (A_BYTES + W_BYTES);
    const char* sw = TRI ? stage_w(buf) : sa + A_BYTES;
    const int c = (KS / 8) * s + lkc;
#pragma unroll
    for (int i = 0; i < TI; i++) fw[rb][i] = *(const bf16x8*)(sw + wrow0 + MS * i * 128 + ((c ^ fwk[i]) << 4));
#pragma unroll
    for (int j = 0; j < TJ; j++) fa[rb][j] = *(const bf16x8*)(sa + arow0 + MS * j * 128 + ((c ^ fak[j]) << 4));
  };

  // One k-tile held in LDS stage `buf`. Every tile but the last ends with the hand-over: wait until
  // tile kt+1 has landed and every wave is done reading stage `buf`, then, while the last MFMAs of
  // tile kt run, refill `buf` with tile kt+2 (PH == 0; the next-to-last tile has nothing left to
  // load, PH == 1) and read the first fragments of tile kt+1. The phases are separate code paths so
  // that the refill needs no branch (the direct-to-LDS loads can then be interleaved with the MFMAs
  // instead of stalling every wave behind the barrier), and so that the compiler never merges paths
  // in front of those MFMAs (at a merge it also waits for the fresh fragment reads).
  // The reads and loads of a k step are spread over its MFMAs: loads over the first half, fragment
  // reads over the first three quarters, leaving the tail of the step to cover their latency.
  constexpr int NM = TI * TJ;
  auto ktile = [&](int kt, auto ph_c) {
    constexpr int PH = decltype(ph_c)::value;
    const int buf = kt & 1;
#pragma unroll
    for (int s = 0; s < BK / KS; s++) {
      const int rb = s & 1;
      const bool seam = s == BK / KS - 1;
      if (!seam) {
        frags(buf, s + 1, rb ^ 1);
      } else if (PH < 2) {
        __builtin_amdgcn_s_waitcnt(0);   // tile kt+1 landed and this wave's reads of `buf` are done
        __syncthreads();                 // ... in every wave: `buf` may be refilled
        if (PH == 0) issue(kt + 2, buf);
        frags(buf ^ 1, 0, rb ^ 1);
      }
#pragma unroll
      for (int i = 0; i < TI; i++)
#pragma unroll
        for (int j = 0; j < TJ; j++)
          acc[i][j] = Mfma<MS>::run(fw[rb][i], fa[rb][j], acc[i][j]);
      if (!seam) sched_step<NM, 0, TI + TJ>();
      else sched_step<NM, PH == 0 ? A_LOADS + W_LOADS : 0, PH < 2 ? TI + TJ : 0>();
    }
  };

  // Epilogue inputs (bias, gate vectors, RoPE table) are requested into registers before the last
  // k-tile, so their memory latency is covered by its MFMAs; after the loop they are written to LDS.
  // Tiles whose inputs exceed the register budget (more than one gate row per thread or four table
  // entries per thread) load them after the loop instead.
  constexpr int NT = NW * 64;
  constexpr int LDS_BYTES = 2 * (A_BYTES + W_BYTES);
  const int rpb = (int)P.cmap.rows_per_batch;
  const int bfirst = m0 / rpb;
  const int nbt = (min(m0 + BM, P.M) - 1) / rpb - bfirst + 1;
  const bool gate_lds = EPI == EPI_RESID && (size_t)(BN + nbt * BN) * 4 <= (size_t)LDS_BYTES;
  const int rope_n = (EPI == EPI_QKV && P.rope_tab) ? P.rope_npos * (P.head_dim >> 1) : 0;
  const bool rope_lds = rope_n > 0 && (size_t)(BN + rope_n) * 4 <= (size_t)LDS_BYTES;
  const bool pre = (!gate_lds || nbt * BN <= NT) && (!rope_lds || rope_n <= 4 * NT);
  // branch-free buffer loads: a lane with nothing to fetch uses an offset past num_records and reads 0
  u16 pre_b = 0;
  float pre_g = 0.f, pre_r[4] = {0.f, 0.f, 0.f, 0.f};
  auto prefetch_epi = [&]() {
    if (!pre) return;
    const uint32_t OOB = 0x80000000u;
    const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
        P.bias ? (void*)P.bias : (void*)P.W, (short)0, P.bias ? P.N * 2 : 0, 0x00020000);
    pre_b = __builtin_amdgcn_raw_buffer_load_b16(rb, tid < BN ? (uint32_t)(n0 + tid) * 2u : OOB, 0, 0);
    if (gate_lds) {
      const __amdgpu_buffer_rsrc_t rg = __builtin_amdgcn_make_buffer_rsrc((void*)P.gate, (short)0, 0x7fffffff, 0x00020000);
      const int bb = tid / BN, nn = tid - bb * BN;
      const bool ok = bb < nbt && n0 + nn < P.N;
      pre_g = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
          rg, ok ? (uint32_t)(((int64_t)(bfirst + bb) * P.gate_bstride + n0 + nn) * 4) : OOB, 0, 0));
    }
    if (rope_lds) {
      const __amdgpu_buffer_rsrc_t rr = __builtin_amdgcn_make_buffer_rsrc((void*)P.rope_tab, (short)0, rope_n * 4, 0x00020000);
#pragma unroll
      for (int r = 0; r < 4; r++)
        pre_r[r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rr, (uint32_t)(tid + r * NT) * 4u, 0, 0));
    }
  };

  if constexpr (TRI) {
    // k-tile kt. First step: refill A stage (kt+2) % 3 with tile kt+2 (that stage last held tile
    // kt-1, whose reads ended before the previous barrier). Last step: wait for tile kt+1 (the A
    // loads of tile kt+2, issued last, may still be in flight: vmcnt(A_LOADS)), barrier, then
    // refill W stage kt % 2 with tile kt+2 and read tile kt+1's first fragments.
    // Issue priority between two barriers runs 3, 2 (halves of the last step), 1, 0 (halves of
    // the next tile's first step): a wave that has run ahead yields the matrix pipe to the other
    // wave of its SIMD, so both reach the barrier together.
    auto ktile3 = [&](int kt, auto ph_c) {
      constexpr int PH = decltype(ph_c)::value;   // 0, 1: refill tile kt+2; 2: none; 3: last tile
#pragma unroll
      for (int s = 0; s < BK / KS; s++) {
        const int rb = s & 1;
        const bool seam = s == BK / KS - 1;
        if (!seam) {
          __builtin_amdgcn_s_setprio(1);
          frags(kt, s + 1, rb ^ 1);
          if (PH <= 1) issue_a(kt + 2);
        } else if (PH < 3) {
          if (PH < 2) __builtin_amdgcn_s_waitcnt(0x0070 | A_LOADS);   // vmcnt(A_LOADS) lgkmcnt(0)
          else __builtin_amdgcn_s_waitcnt(0);
          __syncthreads();
          __builtin_amdgcn_s_setprio(3);
          if (PH <= 1) issue_w(kt + 2);
          frags(kt + 1, 0, rb ^ 1);
        }
        // the step's MFMAs in two halves; the priority drops between them (a scheduling boundary,
        // so the step's reads and loads are placed among the first half's MFMAs)
#pragma unroll
        for (int i = 0; i < TI / 2; i++)
#pragma unroll
          for (int j = 0; j < TJ; j++)
            acc[i][j] = Mfma<MS>::run(fw[rb][i], fa[rb][j], acc[i][j]);
        if (!seam) sched_step<NM / 2, PH <= 1 ? A_LOADS : 0, TI + TJ>();
        else sched_step<NM / 2, PH <= 1 ? W_LOADS : 0, PH < 3 ? TI + TJ : 0>();
        if (seam) __builtin_amdgcn_s_setprio(2);
        else __builtin_amdgcn_s_setprio(0);
#pragma unroll
        for (int i = TI / 2; i < TI; i++)
#pragma unroll
          for (int j = 0; j < TJ; j++)
            acc[i][j] = Mfma<MS>::run(fw[rb][i], fa[rb][j], acc[i][j]);
      }
    };
    issue_a(0);
    issue_w(0);
    if (nk > 1) issue_a(1);
    if (nk > 1) __builtin_amdgcn_s_waitcnt(0x0070 | A_LOADS);
    else __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (nk > 1) issue_w(1);
    frags(0, 0, 0);
    for (int kt = 0; kt + 3 < nk; kt++) ktile3(kt, std::integral_constant<int, 0>());
    if (nk >= 3) ktile3(nk - 3, std::integral_constant<int, 1>());
    if (nk >= 2) ktile3(nk - 2, std::integral_constant<int, 2>());
    prefetch_epi();
    ktile3(nk - 1, std::integral_constant<int, 3>());
    __builtin_amdgcn_s_setprio(0);
  } else {
    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (nk > 1) issue(1, 1);
    frags(0, 0, 0);
    for (int kt = 0; kt + 2 < nk; kt++) ktile(kt, std::integral_constant<int, 0>());
    if (nk >= 2) ktile(nk - 2, std::integral_constant<int, 1>());
    prefetch_epi();
    ktile(nk - 1, std::integral_constant<int, 2>());
  }

  // ---- epilogue: bias, gate vectors and the RoPE table are staged in LDS once per tile ----
  // accumulator (i, j), register r = 4 g + q (q = 0..3):
  //   MS = 32: n = 32 i + 8 g + 4 (lane / 32) + q, m = 32 j + lane % 32
  //   MS = 16: n = 16 i + 4 (lane / 16) + q,        m = 16 j + lane % 16
  constexpr int NG = NACC / 4;
  // MS = 16 with bf16 output: blocks i and i + 1 of a row group (32 adjacent columns) are finished
  // together and regrouped with v_permlane16_swap, which exchanges lanes 16-31 of one register with
  // lanes 0-15 of another (and 48-63 with 32-47). Lane group g = lane / 16 then holds the 8 adjacent
  // columns 32 p + 16 (g & 1) + 8 (g >> 1) of pair p, stored with one 16-byte store. A CU issues a
  // store of 16 rows x 32 B (the accumulator layout) in ~74 cycles and one of 16 rows x 64 B in ~20,
  // and with 256 stores per tile that issue time, not HBM, bounded the epilogue. The paired layout
  // needs 16-byte aligned output rows; otherwise the accumulator layout is stored as it is.
  constexpr bool PAIRS = MS == 16 && !OUTF32;
  static_assert(!PAIRS || TI % 2 == 0, "the paired store joins blocks 2p and 2p + 1");
  const bool pairs = PAIRS && (P.N & 7) == 0 && ((uintptr_t)P.C & 15) == 0 &&
                     ((P.cmap.batch_stride | P.cmap.row_stride | P.cmap.offset) & 7) == 0;
  const int pair_col = 16 * (lkc & 1) + 8 * (lkc >> 1);
  // MS = 16: the residual values of this wave's whole sub-tile (64 registers, free now that the
  // fragment registers are dead) are requested at once, before the staging barriers, so their memory
  // latency is paid once per tile and overlaps the staging. xq[j][p] holds blocks (2p, j) and
  // (2p + 1, j): in the paired layout as loaded (one 16-byte load), else as two 8-byte loads in the
  // accumulator layout.
  constexpr bool XALL = EPI == EPI_RESID && MS == 16;
  static_assert(!XALL || PAIRS, "the residual preload assumes paired blocks");
  uint4 xq[XALL ? TJ : 1][XALL ? TI / 2 : 1];
  if constexpr (XALL) {
    // buffer loads, so that no load sits in a branch: a conditional load leaves the compiler unable to
    // count the loads in flight, and it then waits for every earlier memory operation (stores
    // included) before each use
    const uint32_t OOB = 0x80000000u;
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(P.C, (short)0, 0x7fffffff, 0x00020000);
    if (pairs) {
#pragma unroll
      for (int j = 0; j < TJ; j++) {
        const int m = m0 + wm * WTM + MS * j + frow;
        const uint32_t roff = m < P.M ? (uint32_t)(row_epi(P, m).off * 2) : OOB;
#pragma unroll
        for (int p = 0; p < TI / 2; p++) {
          const int c = n0 + wn * WTN + 32 * p + pair_col;
          const uint32_t off = (m < P.M && c < P.N) ? roff + (uint32_t)c * 2u : OOB;
          xq[j][p] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rc, off, 0, 0));
        }
      }
    } else {
#pragma unroll
      for (int j = 0; j < TJ; j++) {
        const int m = m0 + wm * WTM + MS * j + frow;
        const uint32_t roff = m < P.M ? (uint32_t)(row_epi(P, m).off * 2) : OOB;
#pragma unroll
        for (int p = 0; p < TI / 2; p++) {
          uint2 h[2];
#pragma unroll
          for (int e = 0; e < 2; e++) {
            const int n = n0 + wn * WTN + MS * (2 * p + e) + 4 * lkc;
            const uint32_t off = (m < P.M && n < P.N) ? roff + (uint32_t)n * 2u : OOB;
            h[e] = __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(rc, off, 0, 0));
          }
          xq[j][p] = make_uint4(h[0].x, h[0].y, h[1].x, h[1].y);
        }
      }
    }
  }
  __syncthreads();   // every wave is done with the operand tiles
  float* s_bias = (float*)smem;                       // [BN]
  float* s_gate = s_bias + BN;                        // [nbt][BN]
  float* s_rope = s_bias + BN;                        // [npos][head_dim/4][2] (QKV only)
  if (pre) {
    if (tid < BN) s_bias[tid] = to_f32(pre_b);
    if (gate_lds && tid < nbt * BN) s_gate[tid] = pre_g;
    if (rope_lds) {
#pragma unroll
      for (int r = 0; r < 4; r++)
        if (tid + r * NT < rope_n) s_rope[tid + r * NT] = pre_r[r];
    }
  } else {
    for (int q = tid; q < BN; q += NT)
      s_bias[q] = (P.bias && n0 + q < P.N) ? to_f32(((const u16*)P.bias)[n0 + q]) : 0.f;
    if (gate_lds)
      for (int q = tid; q < nbt * BN; q += NT) {
        int bb = q / BN, nn = q - bb * BN;
        s_gate[q] = n0 + nn < P.N ? P.gate[(int64_t)(bfirst + bb) * P.gate_bstride + n0 + nn] : 0.f;
      }
    if (rope_lds)
      for (int q = tid; q < rope_n; q += NT) s_rope[q] = P.rope_tab[q];
  }
  __syncthreads();

  // The store loop reads the gate vectors and the RoPE table either from LDS (STAGED) or, for tiles
  // whose inputs did not fit the staging area, from global memory. The two are separate instances:
  // a pointer that may point to either is a flat address, and a flat load makes the compiler wait
  // for every store issued before it.
  const bool rope_on = EPI == EPI_QKV && P.rope_tab != nullptr;
  const int rope_cols = 2 * P.hidden, head_dim = P.head_dim;
  auto store_tile = [&](auto staged_c) {
    constexpr bool STAGED = decltype(staged_c)::value;
#pragma unroll
    for (int j = 0; j < TJ; j++) {
      int m = m0 + wm * WTM + MS * j + frow;
      if (m >= P.M) continue;
      const RowEpi R = row_epi(P, m);
      const int bt = m / rpb - bfirst;
      // residual rows: prefetch the 32-column block i+1 while block i is finished
      uint2 xr[2][4];
      auto load_x = [&](int i, int slot) {
#pragma unroll
        for (int g = 0; g < NG; g++) {
          int n = n0 + wn * WTN + MS * i + 8 * g + 4 * lkc;
          if (EPI == EPI_RESID && n < P.N) xr[slot][g] = *(const uint2*)((const u16*)P.C + R.off + n);
        }
      };
      if (EPI == EPI_RESID && !XALL) load_x(0, 0);
#pragma unroll
      for (int i = 0; i < TI; i++) {
        if (EPI == EPI_RESID && !XALL && i + 1 < TI) load_x(i + 1, (i + 1) & 1);
#pragma unroll
        for (int g = 0; g < NG; g++) {
          int nl = wn * WTN + MS * i + 8 * g + 4 * lkc;   // column inside the tile
          int n = n0 + nl;
          if (n >= P.N) continue;
          float v[4] = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]};
          float4 bv = *(const float4*)(s_bias + nl);
          v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
          if (EPI == EPI_GELU) {
#pragma unroll
            for (int q = 0; q < 4; q++) v[q] = gelu_tanh_f(v[q]);
          }
          if (EPI == EPI_RESID) {
            float4 gv = STAGED ? *(const float4*)(s_gate + bt * BN + nl) : *(const float4*)(P.gate + R.gate + n);
            uint2 u = xr[i & 1][g];
            if constexpr (XALL) {
              const uint4 q = xq[j][i >> 1];
              u = (i & 1) ? make_uint2(q.z, q.w) : make_uint2(q.x, q.y);
            }
            v[0] = fmaf(gv.x, v[0], __uint_as_float(u.x << 16));
            v[1] = fmaf(gv.y, v[1], __uint_as_float(u.x & 0xffff0000u));
            v[2] = fmaf(gv.z, v[2], __uint_as_float(u.y << 16));
            v[3] = fmaf(gv.w, v[3], __uint_as_float(u.y & 0xffff0000u));
          }
          if (EPI == EPI_QKV && rope_on && n < rope_cols) {
            int dd = n & (head_dim - 1);
            int hh = head_dim >> 1;
            int pos = dd < hh ? R.rpos : R.cpos;
            int pr = (dd & (hh - 1)) >> 1;
            int ti = (pos * (head_dim >> 2) + pr) * 2;
            float4 t = STAGED ? *(const float4*)(s_rope + ti) : *(const float4*)(P.rope_tab + ti);
            float a0 = v[0], b0 = v[1], a1 = v[2], b1 = v[3];
            v[0] = a0 * t.x - b0 * t.y;
            v[1] = a0 * t.y + b0 * t.x;
            v[2] = a1 * t.z - b1 * t.w;
            v[3] = a1 * t.w + b1 * t.z;
          }
          if (OUTF32) store4<float>((float*)P.C + R.off + n, v);
          else store4<u16>((u16*)P.C + R.off + n, v);
        }
      }
    }
  };
  // The paired store: the same arithmetic per accumulator block as store_tile, then the regrouping
  // swap on the packed bf16 pairs and one 16-byte store per pair of blocks. The residual values arrive
  // in the paired layout and go through the same swap (it is its own inverse) before use.
  auto store_pairs = [&](auto staged_c) {
    constexpr bool STAGED = decltype(staged_c)::value;
    if constexpr (PAIRS) {
#pragma unroll
      for (int j = 0; j < TJ; j++) {
        const int m = m0 + wm * WTM + MS * j + frow;
        if (m >= P.M) continue;   // the swap partners (lanes l and l ^ 16) share the row m
        const RowEpi R = row_epi(P, m);
        const int bt = m / rpb - bfirst;
#pragma unroll
        for (int p = 0; p < TI / 2; p++) {
          uint4 xr = make_uint4(0u, 0u, 0u, 0u);
          if constexpr (XALL) {
            xr = xq[j][p];
            swap16(xr.x, xr.z);
            swap16(xr.y, xr.w);
          }
          uint32_t w[2][2];
#pragma unroll
          for (int e = 0; e < 2; e++) {
            const int i = 2 * p + e;
            const int nl = wn * WTN + MS * i + 4 * lkc;   // column inside the tile
            const int n = n0 + nl;
            float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
            float4 bv = *(const float4*)(s_bias + nl);
            v[0] += bv.x; v[1] += bv.y; v[2] += bv.z; v[3] += bv.w;
            if (EPI == EPI_GELU) {
#pragma unroll
              for (int q = 0; q < 4; q++) v[q] = gelu_tanh_f(v[q]);
            }
            if (EPI == EPI_RESID) {
              float4 gv = make_float4(0.f, 0.f, 0.f, 0.f);
              if (STAGED) gv = *(const float4*)(s_gate + bt * BN + nl);
              else if (n < P.N) gv = *(const float4*)(P.gate + R.gate + n);
              const uint32_t u0 = e ? xr.z : xr.x, u1 = e ? xr.w : xr.y;
              v[0] = fmaf(gv.x, v[0], __uint_as_float(u0 << 16));
              v[1] = fmaf(gv.y, v[1], __uint_as_float(u0 & 0xffff0000u));
              v[2] = fmaf(gv.z, v[2], __uint_as_float(u1 << 16));
              v[3] = fmaf(gv.w, v[3], __uint_as_float(u1 & 0xffff0000u));
            }
            if (EPI == EPI_QKV && rope_on && n < rope_cols) {
              int dd = n & (head_dim - 1);
              int hh = head_dim >> 1;
              int pos = dd < hh ? R.rpos : R.cpos;
              int pr = (dd & (hh - 1)) >> 1;
              int ti = (pos * (head_dim >> 2) + pr) * 2;
              float4 t = STAGED ? *(const float4*)(s_rope + ti) : *(const float4*)(P.rope_tab + ti);
              float a0 = v[0], b0 = v[1], a1 = v[2], b1 = v[3];
              v[0] = a0 * t.x - b0 * t.y;
              v[1] = a0 * t.y + b0 * t.x;
              v[2] = a1 * t.z - b1 * t.w;
              v[3] = a1 * t.w + b1 * t.z;
            }
            w[e][0] = pack_bf16x2(v[0], v[1]);
            w[e][1] = pack_bf16x2(v[2], v[3]);
          }
          swap16(w[0][0], w[1][0]);
          swap16(w[0][1], w[1][1]);
          const int c = n0 + wn * WTN + 32 * p + pair_col;
          if (c < P.N) *(uint4*)((u16*)P.C + R.off + c) = make_uint4(w[0][0], w[0][1], w[1][0], w[1][1]);
        }
      }
    }
  };
  const bool staged = (EPI != EPI_RESID || gate_lds) && (!rope_on || rope_lds);
  // XALL: every residual load has landed before the first store. The compiler cannot order stores
  // against loads on this counter, so inside the loop it would instead wait for earlier stores.
  if constexpr (XALL) __builtin_amdgcn_s_waitcnt(0);
  if (pairs) {
    if (staged) store_pairs(std::true_type());
    else store_pairs(std::false_type());
  } else {
    if (staged) store_tile(std::true_type());
    else store_tile(std::false_type());
  }
#endif
}

template <int BM, int BN, int WM, int WN, int EPI, bool OUTF32, int MS, bool TRI = false>
static hipError_t launch_bf16(const GemmPair& pr, hipStream_t s) {
  int tiles[2] = {0, 0};
  for (int i = 0; i < pr.nprob; i++)
    if (pr.p[i].M > 0 && pr.p[i].N > 0) tiles[i] = cdiv(pr.p[i].M, BM) * cdiv(pr.p[i].N, BN);
  int total = tiles[0] + tiles[1];
  if (total == 0) return hipSuccess;
  size_t lds = TRI ? (size_t)(2 * BN + 3 * BM) * 64 * 2 : 2 * (size_t)(BM + BN) * 64 * 2;
  // The dynamic-LDS limit is raised once per device and kernel instance. Two host threads may reach
  // this at once; setting the attribute twice is harmless, and the flag is an atomic so the check
  // itself is race-free.
  static std::atomic<bool> attr_set[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) dev = 0;
  if (lds > 65536 && (dev < 0 || dev >= 64 || !attr_set[dev].load(std::memory_order_acquire))) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_kernel<BM, BN, WM, WN, EPI, OUTF32, MS, TRI>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64) attr_set[dev].store(true, std::memory_order_release);
  }
  int grid = 8 * cdiv(total, 8);
  gemm_bf16_kernel<BM, BN, WM, WN, EPI, OUTF32, MS, TRI><<<grid, WM * WN * 64, lds, s>>>(pr, tiles[0], total);
  return hipGetLastError();
}

// Compute units of the current device (one 256 x 256 workgroup fills a CU: 160 KB of LDS and the
// whole register file), read once per device.
static int cu_count() {
  static std::atomic<int> cus[64] = {};   // 0 = not read yet; concurrent first reads store the same value
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

template <int EPI, bool OUTF32>
static hipError_t dispatch_bf16(const GemmPair& pr, hipStream_t s) {
  int maxn = 0;
  int64_t big_tiles = 0;
  for (int i = 0; i < pr.nprob; i++) {
    maxn = std::max(maxn, pr.p[i].N);
    big_tiles += (int64_t)cdiv(pr.p[i].M, 256) * cdiv(pr.p[i].N, 256);
  }
  if (maxn <= 64) return launch_bf16<64, 64, 2, 2, EPI, OUTF32, 32>(pr, s);
  // 128 x 128 tiles (4 waves, two workgroups per CU) or 256 x 256 tiles (8 waves, one per CU): the
  // one with fewer estimated rounds, a round of 2 x CUs small tiles costing C128 of a large round
  // (a quarter of the flops per tile, at lower MFMA efficiency)
  {
    constexpr double C128 = 0.71;
    const int64_t cus = cu_count();
    int64_t small_tiles = 0;
    for (int i = 0; i < pr.nprob; i++) small_tiles += (int64_t)cdiv(pr.p[i].M, 128) * cdiv(pr.p[i].N, 128);
    const double big = (double)((big_tiles + cus - 1) / cus);
    const double small = C128 * (double)((small_tiles + 2 * cus - 1) / (2 * cus));
    if (small < big) return launch_bf16<128, 128, 2, 2, EPI, OUTF32, 32>(pr, s);
  }
  // large problems: 8 waves of 64x128 on 16x16x32 MFMAs (measured 3-7% faster than 32x32x16 here),
  // with three A stages, so the activation rows are requested two k-tiles ahead (in the denoise step
  // every block's weights and most activation panels arrive cold from HBM).
  //
  // Every CU runs one 256 x 256 tile at a time, so a launch takes ceil(tiles / CUs) rounds of equal
  // length. When the image and text problems together leave the last round partly empty, the text
  // problem can instead run as a second launch of 256 x 192 tiles: with 4096 text rows and 3072 or
  // 9216 output features that divides into whole rounds. A round of 256 x 192 tiles was measured at
  // 0.80-0.83 of a 256 x 256 round (17% more operand bytes per flop than the 0.75 of the flops), so
  // the split is taken when ceil(t_img / CUs) + 0.83 ceil(t_txt' / CUs) rounds beat
  // ceil((t_img + t_txt) / CUs).
  if (pr.nprob == 2 && pr.p[0].M > 0 && pr.p[1].M > 0 && pr.p[0].N > 0 && pr.p[1].N > 0) {
    const int64_t cus = cu_count();
    const int64_t t0 = (int64_t)cdiv(pr.p[0].M, 256) * cdiv(pr.p[0].N, 256);
    const int64_t t1 = (int64_t)cdiv(pr.p[1].M, 256) * cdiv(pr.p[1].N, 256);
    const int64_t t1n = (int64_t)cdiv(pr.p[1].M, 256) * cdiv(pr.p[1].N, 192);
    const double merged = (double)((t0 + t1 + cus - 1) / cus);
    const double split = (double)((t0 + cus - 1) / cus) + 0.83 * (double)((t1n + cus - 1) / cus);
    if (split < merged) {
      GemmPair a = pr, b = pr;
      a.nprob = 1;
      b.nprob = 1;
      b.p[0] = pr.p[1];
      hipError_t e = launch_bf16<256, 256, 4, 2, EPI, OUTF32, 16, true>(a, s);
      if (e != hipSuccess) return e;
      return launch_bf16<256, 192, 4, 2, EPI, OUTF32, 16, true>(b, s);
    }
  }
  return launch_bf16<256, 256, 4, 2, EPI, OUTF32, 16, true>(pr, s);
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
    if (m < P.M && n < P.N) epilogue4<EPI, float, float>(P, row_epi(P, m), n, acc[i]);
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
