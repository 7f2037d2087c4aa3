// Joint non-causal attention on gfx950.
//
// bf16 path (head_dim 64 or 128): flash-style, one workgroup = 4 waves = 128
// queries of one (sample, head); K/V tiles of 64 keys staged in LDS and shared
// by the 4 waves; online softmax in the exp2 domain with fp32 statistics.
//   * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16:
//     operand A = 32 keys (K rows from LDS), operand B = 32 queries (Q rows held
//     in registers for the whole loop). Each lane then owns ONE query column
//     and 16 of its 32 keys per block; the other 16 sit in lane^32, so the row
//     max and row sum need in-lane reductions plus one exchange with lane^32.
//   * O^T = V^T P^T: P^T is consumed straight from the score registers (rounded
//     to bf16) as operand B; the key order inside a 16-key MFMA step is the
//     order the score accumulator already has, and operand A (V^T) is read in
//     that same key order from a transposed V tile in LDS (two ds_read_b64).
//   * K rows in LDS are 16-byte chunks XOR-swizzled by key, V^T rows padded by
//     4 elements, so fragment reads are free of bank conflicts; the fragments of
//     the next MFMA step are read while the current step's MFMAs run.
//   * Workgroups are dispatched round-robin over the 8 XCDs; each XCD gets a
//     contiguous range of (sample, head, query block) tiles, so the query blocks
//     of one (sample, head) read its K/V through the same L2.
// fp32 path: one thread per query, K/V tiles in LDS (small configurations).
#include "internal.h"

namespace dit {

template <int D>
__global__ void __launch_bounds__(256, 2) attn_fwd_bf16(AttnArgs a) {
  constexpr int QB = 128, KB = 64;
  constexpr int CH = D / 8;            // 16-byte chunks per K row
  constexpr int VT = KB + 4;           // padded V^T row (keys)
  constexpr int NDB = D / 32;          // 32-dim output blocks
  constexpr int NKS = D / 16;          // 16-dim steps of QK^T
  __shared__ __attribute__((aligned(16))) u16 sK[2][KB * D];
  __shared__ __attribute__((aligned(16))) u16 sVt[2][D * VT];

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

  // tile loader: KB*CH chunks of K and of V, (KB*CH)/256 per thread each
  constexpr int LPT = KB * CH / 256;
  uint4 kreg[LPT], vreg[LPT];
  auto gload = [&](int kt) {
#pragma unroll
    for (int i = 0; i < LPT; i++) {
      int idx = tid + 256 * i;
      int key = idx % KB, c = idx / KB;   // consecutive lanes -> consecutive keys
      int gk = kt * KB + key;
      if (gk < S) {
        kreg[i] = *(const uint4*)(Kg + (int64_t)gk * a.qs_s + c * 8);
        vreg[i] = *(const uint4*)(Vg + (int64_t)gk * a.qs_s + c * 8);
      } else {
        kreg[i] = make_uint4(0, 0, 0, 0);
        vreg[i] = make_uint4(0, 0, 0, 0);
      }
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LPT; i++) {
      int idx = tid + 256 * i;
      int key = idx % KB, c = idx / KB;
      int slot = c ^ (key % CH);
      *(uint4*)(&sK[buf][key * D + slot * 8]) = kreg[i];
      uint32_t w[4] = {vreg[i].x, vreg[i].y, vreg[i].z, vreg[i].w};
#pragma unroll
      for (int e = 0; e < 4; e++) {
        sVt[buf][(c * 8 + 2 * e) * VT + key] = (u16)(w[e] & 0xffff);
        sVt[buf][(c * 8 + 2 * e + 1) * VT + key] = (u16)(w[e] >> 16);
      }
    }
  };

  f32x16 o[NDB];
#pragma unroll
  for (int i = 0; i < NDB; i++)
#pragma unroll
    for (int r = 0; r < 16; r++) o[i][r] = 0.f;
  const float c = a.scale * 1.4426950408889634f;  // fold log2(e) into the scale
  float m_run = -INFINITY, l_run = 0.f;

  const int nt = cdiv(S, KB);
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nt; kt++) {
    const int buf = kt & 1;
    if (kt + 1 < nt) gload(kt + 1);   // next tile in flight during this tile's math

    // S^T blocks: keys 32 kb + 8(r/4) + 4 half + r%4 of this lane's query.
    // The KB/32 accumulator chains advance together; the K fragments of dim step
    // s+1 are read while the MFMAs of step s run.
    f32x16 st[KB / 32];
#pragma unroll
    for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
      for (int r = 0; r < 16; r++) st[kb][r] = 0.f;
    bf16x8 kf[2][KB / 32];
#pragma unroll
    for (int kb = 0; kb < KB / 32; kb++) {
      const int key = 32 * kb + l32;
      kf[0][kb] = *(const bf16x8*)(&sK[buf][key * D + ((0 + half) ^ (key % CH)) * 8]);
    }
#pragma unroll
    for (int s = 0; s < NKS; s++) {
      if (s + 1 < NKS) {
#pragma unroll
        for (int kb = 0; kb < KB / 32; kb++) {
          const int key = 32 * kb + l32;
          kf[(s + 1) & 1][kb] = *(const bf16x8*)(&sK[buf][key * D + ((2 * (s + 1) + half) ^ (key % CH)) * 8]);
        }
      }
#pragma unroll
      for (int kb = 0; kb < KB / 32; kb++)
        st[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[s & 1][kb], qf[s], st[kb], 0, 0, 0);
    }
    // mask keys past the end (last tile only)
    if ((kt + 1) * KB > S) {
#pragma unroll
      for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
        for (int r = 0; r < 16; r++) {
          int key = kt * KB + 32 * kb + 8 * (r >> 2) + 4 * half + (r & 3);
          if (key >= S) st[kb][r] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
      for (int r = 0; r < 16; r++) mx = fmaxf(mx, st[kb][r]);
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));   // the other 16 keys of each 32-key block
    const float m_new = fmaxf(m_run, mx * c);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
    bf16x8 pf[KB / 32][2];
#pragma unroll
    for (int kb = 0; kb < KB / 32; kb++)
#pragma unroll
      for (int t = 0; t < 2; t++)
#pragma unroll
        for (int j = 0; j < 8; j++) {
          float p = __builtin_amdgcn_exp2f(fmaf(st[kb][8 * t + j], c, -m_new));
          psum += p;
          pf[kb][t][j] = (__bf16)p;
        }
    l_run = fmaf(l_run, alpha, psum);
#pragma unroll
    for (int i = 0; i < NDB; i++)
#pragma unroll
      for (int r = 0; r < 16; r++) o[i][r] *= alpha;

    // O^T[dim][query] += V^T[dim][keys] P^T[keys][query]; the NDB output chains advance
    // together over the KB/16 key steps, V^T fragments of step q+1 read during step q
    bf16x8 vfr[2][NDB];
    auto read_v = [&](int q, int slot) {
      const int kb = q >> 1, t = q & 1;
#pragma unroll
      for (int db = 0; db < NDB; db++) {
        const u16* vrow = &sVt[buf][(32 * db + l32) * VT];
        int k0 = 32 * kb + 16 * t + 4 * half;
        bf16x4 lo = *(const bf16x4*)(vrow + k0);
        bf16x4 hi = *(const bf16x4*)(vrow + k0 + 8);
        vfr[slot][db] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    };
    read_v(0, 0);
#pragma unroll
    for (int q = 0; q < KB / 16; q++) {
      if (q + 1 < KB / 16) read_v(q + 1, (q + 1) & 1);
#pragma unroll
      for (int db = 0; db < NDB; db++)
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfr[q & 1][db], pf[q >> 1][q & 1], o[db], 0, 0, 0);
    }
    if (kt + 1 < nt) {
      sstore(buf ^ 1);   // buffer buf^1 was last read in iteration kt-1, before the barrier below it
    }
    __syncthreads();
  }

  // normalise: full row sum = this lane's part + lane^32's part
  float l_all = l_run + __shfl_xor(l_run, 32, 64);
  const float inv = 1.0f / l_all;
  if (qi < S) {
    u16* orow = (u16*)a.o + (int64_t)b * a.os_b + (int64_t)qi * a.os_s + (int64_t)h * a.os_h;
#pragma unroll
    for (int db = 0; db < NDB; db++)
#pragma unroll
      for (int g = 0; g < 4; g++) {
        int dim = 32 * db + 8 * g + 4 * half;
        uint2 u;
        u.x = (uint32_t)from_f32<u16>(o[db][4 * g] * inv) | ((uint32_t)from_f32<u16>(o[db][4 * g + 1] * inv) << 16);
        u.y = (uint32_t)from_f32<u16>(o[db][4 * g + 2] * inv) | ((uint32_t)from_f32<u16>(o[db][4 * g + 3] * inv) << 16);
        *(uint2*)(orow + dim) = u;
      }
  }
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
