// Causal varlen grouped-query attention backward for gfx950.
//
// The analytic gradient of the forward (exact attention per sequence):
//   P = exp(scale*S - lse), Delta[t] = <dO[t], O[t]>, dP = dO V^T,
//   dS = P * (dP - Delta), dQ = scale * dS K, dK = scale * dS^T Q, dV = P^T dO,
// with dK/dV summed over the local query heads that share a KV head.
//
// Three passes, deterministic (no atomics; every output element is written
// by exactly one lane):
//   preprocess : Delta per (item, head, row), float32, layout of lse.
//   dK/dV      : unit = (item, KV head, 128-key tile); four waves, each owning
//                32 keys whose K and V rows stay in registers.  The unit
//                loops over the query heads of the KV head's group and over
//                64-row query tiles from the diagonal to the end, staging Q
//                and dO in LDS.  S = Q K^T puts a key in each lane, so
//                P and dS (C layout) feed dV^T = dO^T P and dK^T = Q^T dS as
//                B operands; dO^T and Q^T are read from the row-major tiles
//                with ds_read_b64_tr_b16.
//   dQ         : unit = (item, query head, 128-row tile), like the forward:
//                S^T = K Q^T and dP^T = V dO^T put a query row in each lane;
//                dQ^T = K^T dS^T takes dS^T as B operand and K^T from the
//                row-major K tile via transpose reads.
#include "device_common.hpp"
#include "nsp_internal.hpp"

namespace nsp {
namespace {

// ------------------------------------------------------------ preprocess --

// Delta[t] = sum_d dO[t,i,d] * O[t,i,d].  One group of D/8 lanes per D-row of
// the attention layout (row = (item, token, head)).
template <int D, bool O_F32>
__global__ void __launch_bounds__(256) bwd_preprocess_kernel(AttnArgs a, int64_t q_rows) {
  constexpr int LPR = D / 8;                 // lanes per row
  constexpr int RPB = 256 / LPR;             // rows per block
  const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
  const int sub = threadIdx.x % LPR;
  float acc = 0.f;
  int j = 0;
  if (row < q_rows) {
    int lo = 0, hi = a.n_items - 1;          // last item with q_row0 <= row and L > 0
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.items[mid].q_row0 <= row) lo = mid; else hi = mid - 1;
    }
    j = lo;
    const int64_t e = row * D + sub * 8;
    const bf16x8 g = *(const bf16x8 *)((const bf16 *)a.dout + e);
    if constexpr (O_F32) {
      const f32x4 o0 = *(const f32x4 *)((const float *)a.o + e);
      const f32x4 o1 = *(const f32x4 *)((const float *)a.o + e + 4);
#pragma unroll
      for (int x = 0; x < 4; ++x) acc += (float)g[x] * o0[x] + (float)g[x + 4] * o1[x];
    } else {
      const bf16x8 o = *(const bf16x8 *)((const bf16 *)a.o + e);
#pragma unroll
      for (int x = 0; x < 8; ++x) acc += (float)g[x] * (float)o[x];
    }
  }
#pragma unroll
  for (int off = LPR / 2; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
  if (row < q_rows && sub == 0) {
    const ItemDesc it = a.items[j];
    const int64_t r = row - it.q_row0;
    const int64_t t = r / it.hq, i = r % it.hq;
    a.delta[it.lse_off + i * it.L + t] = acc;
  }
}

// -------------------------------------------------------------------- dQ --

template <int D>
struct DqCfg {
  static constexpr int BM = kFwdBM;
  static constexpr int BN = kFwdBN;
  static constexpr int LD = D + 16;
  static constexpr int KS = D / 16;
  static constexpr int MB = D / 32;
  static constexpr int CPR = D / 8;
  static constexpr int CPT = BN * CPR / 256;
};

template <int D, bool G_F32>
__global__ void __launch_bounds__(256) bwd_dq_kernel(AttnArgs a) {
  using C = DqCfg<D>;
  __shared__ __attribute__((aligned(16))) bf16 sK[C::BN * C::LD];
  __shared__ __attribute__((aligned(16))) bf16 sV[C::BN * C::LD];

  const int4 u = a.units[blockIdx.x];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int m0 = u.y * C::BM;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const int64_t qhead = it.q_off + (int64_t)u.z * D;
  const bf16 *Kg = (const bf16 *)a.k + it.kv_off + (int64_t)u.w * D;
  const bf16 *Vg = (const bf16 *)a.v + it.kv_off + (int64_t)u.w * D;

  const int wq0 = m0 + wave * 32;
  const int qrow = wq0 + l32;
  const int qr = min(qrow, L - 1);

  bf16x8 qf[C::KS], gf[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) {
    qf[s] = *(const bf16x8 *)((const bf16 *)a.q + qhead + qr * qs + 16 * s + 8 * h);
    gf[s] = *(const bf16x8 *)((const bf16 *)a.dout + qhead + qr * qs + 16 * s + 8 * h);
  }
  const int64_t srow = it.lse_off + (int64_t)u.z * L + qr;
  const float lse2 = a.lse_in[srow] * kLog2e;
  const float dlt = a.delta[srow];

  f32x16 acc[C::MB];
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) acc[mb] = f32x16{};

  const int n_end = min(L, m0 + C::BM);
  uint4 rk[C::CPT], rv[C::CPT];
  auto gload = [&](int n0) {
#pragma unroll
    for (int c = 0; c < C::CPT; ++c) {
      const int idx = tid + 256 * c;
      const int row = idx / C::CPR, col = idx % C::CPR;
      const int64_t gr = min(n0 + row, L - 1);
      rk[c] = *(const uint4 *)(Kg + gr * ks + col * 8);
      rv[c] = *(const uint4 *)(Vg + gr * ks + col * 8);
    }
  };
  gload(0);

  for (int n0 = 0; n0 < n_end; n0 += C::BN) {
    __syncthreads();
#pragma unroll
    for (int c = 0; c < C::CPT; ++c) {
      const int idx = tid + 256 * c;
      const int row = idx / C::CPR, col = idx % C::CPR;
      *(uint4 *)(sK + row * C::LD + col * 8) = rk[c];
      *(uint4 *)(sV + row * C::LD + col * 8) = rv[c];
    }
    __syncthreads();
    if (n0 + C::BN < n_end) gload(n0 + C::BN);
    if (n0 > wq0 + 31) continue;

    f32x16 s[2] = {f32x16{}, f32x16{}};
    f32x16 dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int st = 0; st < C::KS; ++st) {
        const int off = (kb * 32 + l32) * C::LD + 16 * st + 8 * h;
        s[kb] = mfma32x32x16(*(const bf16x8 *)(sK + off), qf[st], s[kb]);
        dp[kb] = mfma32x32x16(*(const bf16x8 *)(sV + off), gf[st], dp[kb]);
      }
    const bool diag = n0 + C::BN - 1 > wq0;
    bf16x8 db[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = n0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
        float p = fast_exp2(s[kb][i] * a.scale_log2 - lse2);
        if (diag && key > qrow) p = 0.f;
        db[kb * 2 + (i >> 3)][i & 7] = (bf16)(p * (dp[kb][i] - dlt));
      }
    // dQ^T += K^T dS^T
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        bf16x8 ak = lds_tr_operand(sK, C::LD, 16 * kk, 32 * mb, lane);
        acc[mb] = mfma32x32x16(ak, db[kk], acc[mb]);
      }
  }

  if (qrow < L) {
    const int64_t obase = qhead + (int64_t)qrow * qs;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * mb + 8 * gq + 4 * h;
        f32x4 v4 = {acc[mb][4 * gq] * a.scale, acc[mb][4 * gq + 1] * a.scale,
                    acc[mb][4 * gq + 2] * a.scale, acc[mb][4 * gq + 3] * a.scale};
        if constexpr (G_F32) {
          *(f32x4 *)((float *)a.dq + obase + d0) = v4;
        } else {
          bf16x4 b4 = {(bf16)v4[0], (bf16)v4[1], (bf16)v4[2], (bf16)v4[3]};
          *(bf16x4 *)((bf16 *)a.dq + obase + d0) = b4;
        }
      }
  }
}

// ----------------------------------------------------------------- dK/dV --

template <int D>
struct KvCfg {
  static constexpr int BN = kBwdBN;          // keys per unit
  static constexpr int BM = kBwdBM;          // query rows per iteration
  static constexpr int LD = D + 16;
  static constexpr int KS = D / 16;
  static constexpr int MB = D / 32;
  static constexpr int CPR = D / 8;
  static constexpr int CPT = BM * CPR / 256;
};

template <int D, bool G_F32>
__global__ void __launch_bounds__(256) bwd_dkdv_kernel(AttnArgs a) {
  using C = KvCfg<D>;
  __shared__ __attribute__((aligned(16))) bf16 sQ[C::BM * C::LD];
  __shared__ __attribute__((aligned(16))) bf16 sG[C::BM * C::LD];
  __shared__ __attribute__((aligned(16))) float sL[C::BM];
  __shared__ __attribute__((aligned(16))) float sD[C::BM];

  const int4 u = a.units[blockIdx.x];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int n0 = u.y * C::BN;
  const int i_lo = u.z & 0xffff, i_hi = u.z >> 16;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const int64_t kvhead = it.kv_off + (int64_t)u.w * D;

  const int kbase = n0 + wave * 32;           // first key of this wave
  const int key = kbase + l32;                // this lane's key (MFMA column)
  const int kr = min(key, L - 1);

  bf16x8 kf[C::KS], vf[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) {
    kf[s] = *(const bf16x8 *)((const bf16 *)a.k + kvhead + kr * ks + 16 * s + 8 * h);
    vf[s] = *(const bf16x8 *)((const bf16 *)a.v + kvhead + kr * ks + 16 * s + 8 * h);
  }
  f32x16 dk[C::MB], dv[C::MB];
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) { dk[mb] = f32x16{}; dv[mb] = f32x16{}; }

  const int mt0 = n0 / C::BM;                     // first query tile touching the keys
  const int mt_n = (L + C::BM - 1) / C::BM - mt0; // query tiles per head
  const int n_iter = (i_hi - i_lo) * mt_n;

  uint4 rq[C::CPT], rg[C::CPT];
  float rl = 0.f, rd = 0.f;
  auto gload = [&](int itr) {
    const int hd = i_lo + itr / mt_n;
    const int m = (mt0 + itr % mt_n) * C::BM;
    const bf16 *Qh = (const bf16 *)a.q + it.q_off + (int64_t)hd * D;
    const bf16 *Gh = (const bf16 *)a.dout + it.q_off + (int64_t)hd * D;
#pragma unroll
    for (int c = 0; c < C::CPT; ++c) {
      const int idx = tid + 256 * c;
      const int row = idx / C::CPR, col = idx % C::CPR;
      const int64_t gr = min(m + row, L - 1);
      rq[c] = *(const uint4 *)(Qh + gr * qs + col * 8);
      rg[c] = *(const uint4 *)(Gh + gr * qs + col * 8);
    }
    if (tid < C::BM) {
      const int64_t srow = it.lse_off + (int64_t)hd * L + min(m + tid, L - 1);
      rl = a.lse_in[srow] * kLog2e;
      rd = a.delta[srow];
    }
  };
  if (n_iter > 0) gload(0);

  for (int itr = 0; itr < n_iter; ++itr) {
    const int m0 = (mt0 + itr % mt_n) * C::BM;
    __syncthreads();
#pragma unroll
    for (int c = 0; c < C::CPT; ++c) {
      const int idx = tid + 256 * c;
      const int row = idx / C::CPR, col = idx % C::CPR;
      *(uint4 *)(sQ + row * C::LD + col * 8) = rq[c];
      *(uint4 *)(sG + row * C::LD + col * 8) = rg[c];
    }
    if (tid < C::BM) { sL[tid] = rl; sD[tid] = rd; }
    __syncthreads();
    if (itr + 1 < n_iter) gload(itr + 1);
    if (m0 + C::BM - 1 < kbase) continue;   // every row of the tile is before every key

    f32x16 s[2] = {f32x16{}, f32x16{}};
    f32x16 dp[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int st = 0; st < C::KS; ++st) {
        const int off = (mb * 32 + l32) * C::LD + 16 * st + 8 * h;
        s[mb] = mfma32x32x16(*(const bf16x8 *)(sQ + off), kf[st], s[mb]);
        dp[mb] = mfma32x32x16(*(const bf16x8 *)(sG + off), vf[st], dp[mb]);
      }
    const bool mask = (m0 < kbase + 31) || (m0 + C::BM > L);
    bf16x8 pb[4], db[4];
#pragma unroll
    for (int mb = 0; mb < 2; ++mb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const int qq = mb * 32 + 8 * g4 + 4 * h;   // tile-local query row of element 4*g4
        const f32x4 l4 = *(const f32x4 *)(sL + qq);
        const f32x4 d4 = *(const f32x4 *)(sD + qq);
#pragma unroll
        for (int x = 0; x < 4; ++x) {
          const int i = 4 * g4 + x;
          const int q = m0 + qq + x;
          float p = fast_exp2(s[mb][i] * a.scale_log2 - l4[x]);
          if (mask && (q < key || q >= L)) p = 0.f;
          pb[mb * 2 + (i >> 3)][i & 7] = (bf16)p;
          db[mb * 2 + (i >> 3)][i & 7] = (bf16)(p * (dp[mb][i] - d4[x]));
        }
      }
    // dV^T += dO^T P ;  dK^T += Q^T dS
#pragma unroll
    for (int md = 0; md < C::MB; ++md)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        bf16x8 ag = lds_tr_operand(sG, C::LD, 16 * kk, 32 * md, lane);
        dv[md] = mfma32x32x16(ag, pb[kk], dv[md]);
        bf16x8 aq = lds_tr_operand(sQ, C::LD, 16 * kk, 32 * md, lane);
        dk[md] = mfma32x32x16(aq, db[kk], dk[md]);
      }
  }

  if (key < L) {
    const int64_t obase = kvhead + (int64_t)key * ks;
#pragma unroll
    for (int md = 0; md < C::MB; ++md)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * md + 8 * gq + 4 * h;
        f32x4 k4 = {dk[md][4 * gq] * a.scale, dk[md][4 * gq + 1] * a.scale,
                    dk[md][4 * gq + 2] * a.scale, dk[md][4 * gq + 3] * a.scale};
        f32x4 v4 = {dv[md][4 * gq], dv[md][4 * gq + 1], dv[md][4 * gq + 2], dv[md][4 * gq + 3]};
        if constexpr (G_F32) {
          *(f32x4 *)((float *)a.dk + obase + d0) = k4;
          *(f32x4 *)((float *)a.dv + obase + d0) = v4;
        } else {
          *(bf16x4 *)((bf16 *)a.dk + obase + d0) = bf16x4{(bf16)k4[0], (bf16)k4[1], (bf16)k4[2], (bf16)k4[3]};
          *(bf16x4 *)((bf16 *)a.dv + obase + d0) = bf16x4{(bf16)v4[0], (bf16)v4[1], (bf16)v4[2], (bf16)v4[3]};
        }
      }
  }
}

}  // namespace

hipError_t launch_bwd_preprocess(int head_dim, bool o_f32, const AttnArgs &a, int64_t q_rows,
                                 hipStream_t s) {
  if (q_rows == 0) return hipSuccess;
  const int rpb = 256 / (head_dim / 8);
  dim3 grid((unsigned)((q_rows + rpb - 1) / rpb)), block(256);
  if (head_dim == 128) {
    if (o_f32) bwd_preprocess_kernel<128, true><<<grid, block, 0, s>>>(a, q_rows);
    else bwd_preprocess_kernel<128, false><<<grid, block, 0, s>>>(a, q_rows);
  } else {
    if (o_f32) bwd_preprocess_kernel<64, true><<<grid, block, 0, s>>>(a, q_rows);
    else bwd_preprocess_kernel<64, false><<<grid, block, 0, s>>>(a, q_rows);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dq(int head_dim, bool g_f32, const AttnArgs &a, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  dim3 grid(n_units), block(256);
  if (head_dim == 128) {
    if (g_f32) bwd_dq_kernel<128, true><<<grid, block, 0, s>>>(a);
    else bwd_dq_kernel<128, false><<<grid, block, 0, s>>>(a);
  } else {
    if (g_f32) bwd_dq_kernel<64, true><<<grid, block, 0, s>>>(a);
    else bwd_dq_kernel<64, false><<<grid, block, 0, s>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv(int head_dim, bool g_f32, const AttnArgs &a, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  dim3 grid(n_units), block(256);
  if (head_dim == 128) {
    if (g_f32) bwd_dkdv_kernel<128, true><<<grid, block, 0, s>>>(a);
    else bwd_dkdv_kernel<128, false><<<grid, block, 0, s>>>(a);
  } else {
    if (g_f32) bwd_dkdv_kernel<64, true><<<grid, block, 0, s>>>(a);
    else bwd_dkdv_kernel<64, false><<<grid, block, 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace nsp
