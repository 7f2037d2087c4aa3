// Joint non-causal attention on gfx950.
//
// bf16 path (head_dim 64 or 128): flash-style, one workgroup = 4 waves = 128
// queries of one (sample, head); K/V tiles of 64 keys staged in LDS and shared
// by the 4 waves; online softmax in the exp2 domain with fp32 statistics.
//   * K and V tiles go from global memory straight into LDS (buffer loads with the
//     LDS-destination bit), two LDS buffers each. The buffer resource spans exactly
//     this (sample, head)'s rows, so keys past the end read as zeros with no bounds
//     arithmetic. With head_dim 128 a wave's four loads per operand go out as one
//     burst under a single M0 value.
//   * Software pipeline: the step for tile t takes the exponentials of tile t and the
//     score MFMAs of tile t+1 in one instruction stream (neither depends on the
//     other, so the MFMAs issue between the VALU work), then tile t's P V^T. K tiles
//     are therefore requested two tiles ahead and V tiles one ahead.
//   * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
//     operand A = 32 keys (K rows from LDS), operand B = 32 queries (Q rows held
//     in registers for the whole loop). Each lane then owns ONE query column
//     and 16 of its 32 keys per block; the other 16 sit in lane^32, so the row
//     max and row sum need in-lane reductions plus one exchange with lane^32.
//   * O^T = V^T P^T: P^T is consumed straight from the score registers (rounded
//     to bf16) as operand B; the key order inside a 16-key MFMA step is the
//     order the score accumulator already has. Operand A (V^T) comes from the
//     row-major V tile through ds_read_b64_tr_b16, the LDS read that transposes
//     16-bit elements across each group of 16 lanes: lane s of a group points at
//     4 consecutive dims of key k0 + s/4, and lane j of the group receives keys
//     k0..k0+3 of dim j, which is exactly a quarter of an A fragment.
//   * LDS rows are 16-byte chunks XOR-swizzled by row (K: by key mod chunks per
//     row; V: by key mod 4 in steps of a quarter row), so both the K fragment
//     reads and the transposing V reads are free of bank conflicts.
//   * Lazy rescaling: the running max only moves (and the output is only rescaled)
//     when a row's new max exceeds it by more than TAU in the exp2 domain, so
//     probabilities stay below 2^TAU; the normalisation divides by a row sum taken
//     against the same max, so the result is unchanged.
//   * The normalised output leaves through LDS (the K buffers, free after the last
//     step): a wave writes its 32 rows in the accumulator layout and stores them
//     back as whole rows, one 16-byte chunk per lane, instead of 8-byte pieces
//     scattered over 32 rows per store.
//   * Workgroups are dispatched round-robin over the 8 XCDs; each XCD gets a
//     contiguous range of (sample, head, query block) tiles, so the query blocks
//     of one (sample, head) read its K/V through the same L2.
// fp32 path: one thread per query, K/V tiles in LDS (small configurations).
#include "internal.h"

namespace dit {

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));

// Combine the values of lanes l and l ^ 32 through v_permlane32_swap (a VALU exchange of the two
// 32-lane halves) instead of an LDS permute. With both operands v, the swap's two results hold, in
// every lane, v[l] and v[l ^ 32] (which of the two is which depends on the half), so only symmetric
// combinations are formed from them.
__device__ __forceinline__ void half_pair(float v, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}
__device__ __forceinline__ float pair_max(float v) {
  float a, b;
  half_pair(v, a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float pair_sum(float v) {
  float a, b;
  half_pair(v, a, b);
  return a + b;
}

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));

// Four direct-to-LDS loads under one M0 value: destination M0 + 1024 i + 16 lane, global offset
// v[i] + 1024 i (the instruction offset moves both addresses). Issued back to back they hold the
// wave's issue for less than four separately issued loads, each of which sets M0 on its own.
// Inline assembly, so the compiler does not track these loads: the wait before the barrier that
// hands a stage over is the explicit s_waitcnt(0) of the loop.
__device__ __forceinline__ void dma4_b128(u32x4_t rsrc, uint32_t m0v, uint32_t v0, uint32_t v1, uint32_t v2,
                                          uint32_t v3) {
  uint32_t saved;
  asm volatile("s_mov_b32 %0, m0\n\ts_mov_b32 m0, %1\n\ts_nop 0\n\t"
               "buffer_load_dwordx4 %2, %6, 0 offen lds\n\t"
               "buffer_load_dwordx4 %3, %6, 0 offen offset:1024 lds\n\t"
               "buffer_load_dwordx4 %4, %6, 0 offen offset:2048 lds\n\t"
               "buffer_load_dwordx4 %5, %6, 0 offen offset:3072 lds\n\t"
               "s_mov_b32 m0, %0"
               : "=&s"(saved) : "s"(m0v), "v"(v0), "v"(v1), "v"(v2), "v"(v3), "s"(rsrc) : "memory");
}

template <int D>
__global__ void __launch_bounds__(256, 2) attn_fwd_bf16(AttnArgs a) {
  constexpr int QB = 128, KB = 64;
  constexpr int CH = D / 8;            // 16-byte chunks per K/V row
  constexpr int RB = D * 2;            // bytes per K/V row
  constexpr int TILE = KB * RB;        // bytes per K (or V) tile
  constexpr int NDB = D / 32;          // 32-dim output blocks
  constexpr int NKS = D / 16;          // 16-dim steps of QK^T
  constexpr int KPI = 64 / CH;         // rows per 1 KB wave load
  constexpr int LOADS = KB / KPI / 4;  // wave loads per wave per tile, for K and for V each
  constexpr float TAU = 8.f;           // lazy-rescale threshold (log2 units)
  static_assert(LOADS >= 1, "tile too small for 4 waves");
#if defined(__HIP_DEVICE_COMPILE__)  // the buffer-resource builtins exist only in the device pass
  __shared__ __attribute__((aligned(1024))) char smem[4 * TILE];   // [K0][K1][V0][V1]

  // XCD-aware order: workgroup ids go round-robin over the 8 XCDs; give each XCD a
  // contiguous range of (sample, head, query-block) tiles so the query blocks of one
  // (sample, head) share K/V through that XCD's L2.
  const int nqb = cdiv(a.S, QB), per = (nqb * a.H * a.B + 7) / 8;
  const int wid = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
  const int lt = (wid & 7) * per + (wid >> 3);
  if (lt >= nqb * a.H * a.B) return;
  const int qblk = lt % nqb, bh = lt / nqb;
  const int b = bh / a.H, h = bh % a.H;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int half = lane >> 5, l32 = lane & 31;
  const int S = a.S;
  const u16* Q = (const u16*)a.q + (int64_t)b * a.qs_b + (int64_t)h * a.qs_h;
  const u16* Kg = (const u16*)a.k + (int64_t)b * a.qs_b + (int64_t)h * a.qs_h;
  const u16* Vg = (const u16*)a.v + (int64_t)b * a.qs_b + (int64_t)h * a.qs_h;

  // this lane's query and its Q fragments: q[qi][16 s + 8 half + 0..7]
  const int qi = qblk * QB + wave * 32 + l32;
  bf16x8 qf[NKS];
  {
    const u16* qrow = Q + (int64_t)min(qi, S - 1) * a.qs_s;
#pragma unroll
    for (int s = 0; s < NKS; s++) qf[s] = *(const bf16x8*)(qrow + 16 * s + 8 * half);
  }

  // direct-to-LDS loads: wave load i of this wave fills rows R0..R0+KPI-1 of a tile
  // (R0 = (wave * LOADS + i) * KPI); lane -> row R0 + lane / CH, LDS slot lane % CH,
  // which holds global chunk slot ^ swizzle(row)
  const uint32_t rowstride = (uint32_t)(a.qs_s * 2);
  const uint32_t nrec = (uint32_t)((int64_t)(S - 1) * a.qs_s * 2 + RB);
  __amdgpu_buffer_rsrc_t rk = __builtin_amdgcn_make_buffer_rsrc((void*)Kg, (short)0, (int)nrec, 0x00020000);
  __amdgpu_buffer_rsrc_t rv = __builtin_amdgcn_make_buffer_rsrc((void*)Vg, (short)0, (int)nrec, 0x00020000);
  uint32_t koff[LOADS], voff[LOADS];
#pragma unroll
  for (int i = 0; i < LOADS; i++) {
    const int row = (wave * LOADS + i) * KPI + lane / CH, slot = lane % CH;
    koff[i] = row * rowstride + ((slot ^ (row % CH)) << 4);
    voff[i] = row * rowstride + ((slot ^ ((row & 3) * (CH / 4))) << 4);
  }
  // head_dim 128: a wave's share of a K (or V) tile is four consecutive 1 KB blocks, loaded as one burst.
  // Those descriptors start 4 KB early (and span 4 KB more) so that no per-lane offset goes negative.
  const uint64_t k64 = (uint64_t)Kg - 4096, v64 = (uint64_t)Vg - 4096;
  const u32x4_t rk4 = {(uint32_t)k64, (uint32_t)(k64 >> 32) & 0xffffu, nrec + 4096u, 0x00020000u};
  const u32x4_t rv4 = {(uint32_t)v64, (uint32_t)(v64 >> 32) & 0xffffu, nrec + 4096u, 0x00020000u};
  const uint32_t wdst = (uint32_t)(__builtin_amdgcn_readfirstlane(wave) * LOADS * KPI * RB);
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
  auto issue_k = [&](int kt, int buf) {
    const uint32_t base = (uint32_t)(kt * KB) * rowstride;
    if constexpr (LOADS == 4) {
      dma4_b128(rk4, lds0 + buf * TILE + wdst, base + koff[0] + 4096u, base + koff[1] + 3072u, base + koff[2] + 2048u,
                base + koff[3] + 1024u);
    } else {
#pragma unroll
      for (int i = 0; i < LOADS; i++) {
        const int dst = (wave * LOADS + i) * KPI * RB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_ptr_t)(smem + buf * TILE + dst), 16, base + koff[i], 0, 0, 0);
      }
    }
  };
  auto issue_v = [&](int kt, int buf) {
    const uint32_t base = (uint32_t)(kt * KB) * rowstride;
    if constexpr (LOADS == 4) {
      dma4_b128(rv4, lds0 + (2 + buf) * TILE + wdst, base + voff[0] + 4096u, base + voff[1] + 3072u,
                base + voff[2] + 2048u, base + voff[3] + 1024u);
    } else {
#pragma unroll
      for (int i = 0; i < LOADS; i++) {
        const int dst = (wave * LOADS + i) * KPI * RB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_ptr_t)(smem + (2 + buf) * TILE + dst), 16, base + voff[i],
                                                 0, 0, 0);
      }
    }
  };

  // K fragment of key row 32 kb + l32, dim chunk 2 s + half (swizzle key % CH = l32 % CH)
  const int ksw = l32 % CH;
  const int krow = l32 * RB;
  // V^T fragment quarters: lane reads 4 dims (8 bytes) of key 4 half + (lane >> 2) % 4 (+ step
  // offsets); dims 32 db + 16 ((lane >> 4) & 1) + 4 (lane & 3), i.e. chunk
  // 4 db + 2 ((lane >> 4) & 1) + ((lane >> 1) & 1), byte 8 (lane & 1) inside it
  const int vkey = 4 * half + ((lane >> 2) & 3);
  const int vsw = ((lane >> 2) & 3) * (CH / 4);
  int vbase[NDB];
#pragma unroll
  for (int db = 0; db < NDB; db++) {
    const int ch = 4 * db + 2 * ((lane >> 4) & 1) + ((lane >> 1) & 1);
    vbase[db] = vkey * RB + ((ch ^ vsw) << 4) + 8 * (lane & 1);
  }

  f32x16 o[NDB];
#pragma unroll
  for (int i = 0; i < NDB; i++)
#pragma unroll
    for (int r = 0; r < 16; r++) o[i][r] = 0.f;
  const f32x16 zero = {};
  const float c = a.scale * 1.4426950408889634f;  // fold log2(e) into the scale
  float m_run = -INFINITY, l_run = 0.f;

  const int nt = cdiv(S, KB);
  // S^T blocks of a tile: keys 32 kb + 8(r/4) + 4 half + r%4 of this lane's query. The head dims are
  // taken in four groups; a group's K fragments are read just before its MFMAs.
  auto scores = [&](int kt, f32x16* sn) {
    const char* sk = smem + (kt & 1) * TILE;
    constexpr int NS = NKS / 4 > 0 ? NKS / 4 : 1;
#pragma unroll
    for (int g = 0; g < NKS / NS; g++) {
      bf16x8 kf[NS][KB / 32];
#pragma unroll
      for (int s = 0; s < NS; s++)
#pragma unroll
        for (int kb = 0; kb < KB / 32; kb++)
          kf[s][kb] = *(const bf16x8*)(sk + 32 * kb * RB + krow + (((2 * (g * NS + s) + half) ^ ksw) << 4));
#pragma unroll
      for (int s = 0; s < NS; s++)
#pragma unroll
        for (int kb = 0; kb < KB / 32; kb++) {
          const int sg = g * NS + s;
          sn[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s][kb], qf[sg], sg == 0 ? zero : sn[kb], 0, 0, 0);
        }
    }
  };
  // keys past the end of the sequence (last tile only) score -inf; returns this lane's max
  auto mask_max = [&](int kt, f32x16* sn) {
    if ((kt + 1) * KB > S) {
#pragma unroll
      for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
          int key = kt * KB + 32 * kb + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key >= S) sn[kb][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
      for (int r = 0; r < 16; r++) mx = fmaxf(mx, sn[kb][r]);
    return mx;
  };

  // One step of the software pipeline. On entry st holds the scores of tile kt and mx their lane max.
  // The exponentials of tile kt and the score MFMAs of tile kt+1 (NEXT) sit in one instruction stream,
  // so the compiler can issue the one between the other; then tile kt's P V^T runs. K tiles are
  // requested two tiles ahead and V tiles one ahead, each in its own pair of LDS buffers.
  auto step = [&](int kt, f32x16* st, float& mx, f32x16* sn, float& mxn, auto next_c) {
    constexpr bool NEXT = decltype(next_c)::value;
    // every wave is done with K buffer kt&1 (scores of kt, in the previous step) and V buffer
    // (kt+1)&1 (P V^T of kt-1); this wave's loads into the buffers read below have landed
    __syncthreads();
    if (kt + 2 < nt) issue_k(kt + 2, kt & 1);
    const char* sv = smem + (2 + (kt & 1)) * TILE;
    mx = pair_max(mx);   // with the other 16 keys of each 32-key block (lane ^ 32)
    const float mxs = mx * c;
    if (__ballot(mxs > m_run + TAU) != 0) {   // some row's max moved by more than TAU
      const float m_new = fmaxf(m_run, mxs);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int i = 0; i < NDB; i++)
#pragma unroll
        for (int r = 0; r < 16; r++) o[i][r] *= alpha;
    }
    float psum = 0.f;
    bf16x8 pf[KB / 32][2];
#pragma unroll
    for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
      for (int t = 0; t < 2; t++)
#pragma unroll
        for (int j = 0; j < 8; j++) {
          float p = __builtin_amdgcn_exp2f(fmaf(st[kb][8 * t + j], c, -m_run));
          psum += p;
          pf[kb][t][j] = (__bf16)p;
        }
    if constexpr (NEXT) scores(kt + 1, sn);
    l_run += psum;
    // V(kt+1) is requested only now: issued together with K(kt+2) right after the barrier, the
    // eight waves' loads queued behind each other for ~650 cycles per step; here they meet
    // fewer, and still land before the step's final wait
    if (NEXT) issue_v(kt + 1, (kt + 1) & 1);

    // O^T[dim][query] += V^T[dim][keys] P^T[keys][query] over the KB/16 key steps. Step q covers
    // keys 16 q + {4 half + 0..3, 8 + 4 half + 0..3}, the order of the score accumulator.
#pragma unroll
    for (int q = 0; q < KB / 16; q++) {
      bf16x8 vfr[NDB];
#pragma unroll
      for (int db = 0; db < NDB; db++) {
        const char* p0 = sv + 16 * q * RB + vbase[db];
        i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p0));
        i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) i16x4*)(p0 + 8 * RB));
        vfr[db] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
      }
#pragma unroll
      for (int db = 0; db < NDB; db++)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[db], pf[q >> 1][q & 1], o[db], 0, 0, 0);
    }
    if constexpr (NEXT) mxn = mask_max(kt + 1, sn);
    __builtin_amdgcn_s_waitcnt(0);   // this wave's loads of K(kt+2) and V(kt+1) landed
  };

  issue_k(0, 0);
  issue_v(0, 0);
  if (nt > 1) issue_k(1, 1);
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // two score buffers, used alternately (the loop is unrolled by two so that neither is copied)
  f32x16 sa[KB / 32], sb[KB / 32];
  float ma, mb = -INFINITY;
  scores(0, sa);
  ma = mask_max(0, sa);
  int kt = 0;
  for (; kt + 2 < nt; kt += 2) {
    step(kt, sa, ma, sb, mb, std::true_type());
    step(kt + 1, sb, mb, sa, ma, std::true_type());
  }
  if (kt + 1 < nt) {
    step(kt, sa, ma, sb, mb, std::true_type());
    step(kt + 1, sb, mb, sa, ma, std::false_type());
  } else {
    step(kt, sa, ma, sb, mb, std::false_type());
  }

  // normalise: full row sum = this lane's part + lane^32's part
  float l_all = pair_sum(l_run);
  const float inv = 1.0f / l_all;
  // The output tile goes out through LDS: both K buffers are free once every wave has passed the last
  // step's barrier (the last K tile was read by the step before), and each wave uses the 32 rows of
  // that area that hold its own queries, so no further barrier is needed. A wave writes its rows in
  // the accumulator layout (16-byte chunk c of row r at slot c ^ (r mod CH)) and reads them back as
  // whole rows, so that every global store writes complete output rows.
  {
    char* so = smem + wave * 32 * RB;
#pragma unroll
    for (int db = 0; db < NDB; db++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        const int c = 4 * db + g;
        uint2 u;
        u.x = (uint32_t)from_f32<u16>(o[db][4 * g] * inv) | ((uint32_t)from_f32<u16>(o[db][4 * g + 1] * inv) << 16);
        u.y = (uint32_t)from_f32<u16>(o[db][4 * g + 2] * inv) | ((uint32_t)from_f32<u16>(o[db][4 * g + 3] * inv) << 16);
        *(uint2*)(so + l32 * RB + ((c ^ (l32 % CH)) << 4) + 8 * half) = u;
      }
    constexpr int RPI = 64 / CH;   // rows per wave store (CH lanes of 16 bytes per row)
    u16* obase = (u16*)a.o + (int64_t)b * a.os_b + (int64_t)h * a.os_h;
#pragma unroll
    for (int i = 0; i < 32 / RPI; i++) {
      const int r = i * RPI + lane / CH, c = lane % CH;
      const uint4 v = *(const uint4*)(so + r * RB + ((c ^ (r % CH)) << 4));
      const int q = qblk * QB + wave * 32 + r;
      if (q < S) *(uint4*)(obase + (int64_t)q * a.os_s + 8 * c) = v;
    }
  }
#endif
}

// ---------------------------------------------------------------------------
// fp32 attention: one thread per query, online softmax, K/V tiles in LDS
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(64) attn_fwd_f32(AttnArgs a) {
  constexpr int KB = 32;
  __shared__ float sk[KB][D];
  __shared__ float sv[KB][D];
  const int b = blockIdx.z, h = blockIdx.y;
  const int qi = blockIdx.x * 64 + threadIdx.x;
  const float* Q = (const float*)a.q + (int64_t)b * a.qs_b + (int64_t)h * a.qs_h;
  const float* Kg = (const float*)a.k + (int64_t)b * a.qs_b + (int64_t)h * a.qs_h;
  const float* Vg = (const float*)a.v + (int64_t)b * a.qs_b + (int64_t)h * a.qs_h;
  float q[D], acc[D];
  const float* qrow = Q + (int64_t)min(qi, a.S - 1) * a.qs_s;
#pragma unroll
  for (int e = 0; e < D; e++) {
    q[e] = qrow[e] * a.scale;
    acc[e] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  for (int k0 = 0; k0 < a.S; k0 += KB) {
    __syncthreads();
    for (int idx = threadIdx.x; idx < KB * D; idx += 64) {
      int key = idx / D, e = idx % D;
      bool ok = k0 + key < a.S;
      sk[key][e] = ok ? Kg[(int64_t)(k0 + key) * a.qs_s + e] : 0.f;
      sv[key][e] = ok ? Vg[(int64_t)(k0 + key) * a.qs_s + e] : 0.f;
    }
    __syncthreads();
    int nkeys = min(KB, a.S - k0);
    for (int j = 0; j < nkeys; j++) {
      float s = 0.f;
#pragma unroll
      for (int e = 0; e < D; e++) s = fmaf(q[e], sk[j][e], s);
      float mn = fmaxf(m, s);
      float al = __expf(m - mn);
      float p = __expf(s - mn);
      l = l * al + p;
#pragma unroll
      for (int e = 0; e < D; e++) acc[e] = fmaf(acc[e], al, p * sv[j][e]);
      m = mn;
    }
  }
  if (qi < a.S) {
    float* orow = (float*)a.o + (int64_t)b * a.os_b + (int64_t)qi * a.os_s + (int64_t)h * a.os_h;
    float inv = 1.0f / l;
#pragma unroll
    for (int e = 0; e < D; e++) orow[e] = acc[e] * inv;
  }
}

hipError_t attention(const AttnArgs& a, int dtype, hipStream_t s) {
  if (a.B == 0 || a.H == 0 || a.S == 0) return hipSuccess;
  if (dtype == DT_BF16) {
    int nqb = cdiv(a.S, 128);
    int total = nqb * a.H * a.B, per = cdiv(total, 8);
    dim3 grid(nqb, a.H, a.B);
    // the kernel maps linear id -> tile with ceil(total/8) tiles per XCD and ids past the
    // tile count exit; a grid of exactly `total` ids covers every tile when total % 8 == 0
    if (total % 8) grid = dim3(8 * per, 1, 1);
    if (a.d == 128) attn_fwd_bf16<128><<<grid, 256, 0, s>>>(a);
    else attn_fwd_bf16<64><<<grid, 256, 0, s>>>(a);
  } else {
    dim3 grid(cdiv(a.S, 64), a.H, a.B);
    if (a.d == 128) attn_fwd_f32<128><<<grid, 64, 0, s>>>(a);
    else attn_fwd_f32<64><<<grid, 64, 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace dit
