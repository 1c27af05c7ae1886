// Causal varlen grouped-query attention backward for gfx950.
//
// The analytic gradient of the forward (exact attention per sequence):
//   P = exp(scale*S - lse), Delta[t] = <dO[t], O[t]>, dP = dO V^T,
//   dS = P * (dP - Delta), dQ = scale * dS K, dK = scale * dS^T Q, dV = P^T dO,
// with dK/dV summed over the local query heads that share a KV head.
//
// Three passes, deterministic (no atomics; every output element is written
// by exactly one lane):
//   preprocess : Delta per (item, head, row) and lse*log2(e), float32, layout
//                of lse.
//   dK/dV      : unit = (item, KV head, 128-key tile); four waves, each owning
//                32 keys whose K rows stay in registers (the unit's V rows sit
//                in LDS).  The unit loops over the query heads of the KV
//                head's group and over 32-row query tiles from the diagonal to
//                the end; Q, dO, lse2 and Delta tiles stream into double
//                buffered LDS with direct global->LDS loads.  S = Q K^T puts a
//                key in each lane, so P and dS (C layout) feed dV^T = dO^T P
//                and dK^T = Q^T dS as B operands; dO^T and Q^T are read from
//                the row-major tiles with ds_read_b64_tr_b16.
//   dQ         : unit = (item, query head, 128-row tile), like the forward:
//                S^T = K Q^T and dP^T = V dO^T put a query row in each lane;
//                dQ^T = K^T dS^T takes dS^T as B operand and K^T from the
//                row-major K tile via transpose reads; K and V tiles stream
//                into double-buffered LDS.
#include "device_common.hpp"
#include "nsp_internal.hpp"

namespace nsp {
namespace {

// ------------------------------------------------------------ preprocess --

// Delta[t] = sum_d dO[t,i,d] * O[t,i,d], and lse2 = lse * log2(e) (the
// backward works in base 2).  One group of D/8 lanes per D-row of the
// attention layout (row = (item, token, head)).
template <int D, bool O_F32>
__global__ void __launch_bounds__(256) bwd_preprocess_kernel(AttnArgs a, int64_t q_rows) {
  constexpr int LPR = D / 8;                 // lanes per row
  constexpr int RPB = 256 / LPR;             // rows per block
  const int64_t row = (int64_t)blockIdx.x * RPB + threadIdx.x / LPR;
  const int sub = threadIdx.x % LPR;
  float acc = 0.f;
  int j = 0;
  if (row < q_rows) {
    int lo = 0, hi = a.n_items - 1;          // last item with q_row0 <= row
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
    const int64_t o = it.lse_off + i * it.L + t;
    a.delta[o] = acc;
    a.lse2[o] = a.lse_in[o] * kLog2e;
  }
}

// -------------------------------------------------------------------- dQ --

template <int D>
struct DqCfg {
  static constexpr int BM = kFwdBM;
  static constexpr int BN = kFwdBN;
  static constexpr int TILE = BN * D;
  static constexpr int KS = D / 16;
  static constexpr int MB = D / 32;
};

template <int D>
struct DqState {
  bf16x8 qf[D / 16];   // Q^T  (B operand: column = query row, k = head_dim)
  bf16x8 gf[D / 16];   // dO^T (B operand)
  f32x16 acc[D / 32];  // dQ^T (row = head_dim, column = query row)
  float lse2, dlt;
};

// One 64-key tile, in two 32-key halves (to bound live registers):
// S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - Delta), dQ^T += K^T dS^T
// (K^T read from the row-major K tile with transpose reads).
template <int D>
__device__ __forceinline__ void dq_tile(DqState<D> &st, const bf16 *sK, const bf16 *sV, int n0, int wq0, int qrow,
                                        int lane, float c) {
  constexpr int KS = D / 16, MB = D / 32;
  const int l32 = lane & 31, h = lane >> 5;
  const bool diag = n0 + kFwdBN - 1 > wq0;   // tile straddles this wave's diagonal
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) {
    f32x16 s = f32x16{}, p = f32x16{};
#pragma unroll
    for (int k = 0; k < KS; ++k) {
      const int o = tile_off<D>(32 * kb + l32, 16 * k + 8 * h);
      s = mfma32x32x16(*(const bf16x8 *)(sK + o), st.qf[k], s);
      p = mfma32x32x16(*(const bf16x8 *)(sV + o), st.gf[k], p);
    }
    if (diag) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int key = n0 + 32 * kb + 8 * (i >> 2) + 4 * h + (i & 3);
        if (key > qrow) s[i] = -INFINITY;
      }
    }
    bf16x8 db[2];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const float e = fast_exp2(s[i] * c - st.lse2);
      db[i >> 3][i & 7] = (bf16)(e * (p[i] - st.dlt));
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
        st.acc[mb] = mfma32x32x16(lds_tr_operand<D>(sK, 32 * kb + 16 * kk, 32 * mb, lane), db[kk], st.acc[mb]);
  }
}

template <int D, bool G_F32>
__global__ void __launch_bounds__(256, 2) bwd_dq_kernel(AttnArgs a) {
  using C = DqCfg<D>;
  __shared__ __attribute__((aligned(16))) bf16 sK0[C::TILE];
  __shared__ __attribute__((aligned(16))) bf16 sV0[C::TILE];
  __shared__ __attribute__((aligned(16))) bf16 sK1[C::TILE];
  __shared__ __attribute__((aligned(16))) bf16 sV1[C::TILE];

  const int4 u = a.units[blockIdx.x];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int m0 = u.y * C::BM;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const int64_t qhead = it.q_off + (int64_t)u.z * D;
  const TileLoader<D, C::BN> ldK((const bf16 *)a.k + it.kv_off + (int64_t)u.w * D, ks, wave, lane);
  const TileLoader<D, C::BN> ldV((const bf16 *)a.v + it.kv_off + (int64_t)u.w * D, ks, wave, lane);

  const int wq0 = m0 + wave * 32;
  const int qrow = wq0 + l32;
  const int n_end = min(L, m0 + C::BM);
  const int n_tiles = (n_end + C::BN - 1) / C::BN;
  const int wave_tiles = min(n_tiles, (wq0 + 31) / C::BN + 1);

  ldK.load(sK0, 0, L);
  ldV.load(sV0, 0, L);

  DqState<D> st;
  {
    const int64_t r = qhead + (int64_t)min(qrow, L - 1) * qs + 8 * h;
#pragma unroll
    for (int k = 0; k < C::KS; ++k) {
      st.qf[k] = *(const bf16x8 *)((const bf16 *)a.q + r + 16 * k);
      st.gf[k] = *(const bf16x8 *)((const bf16 *)a.dout + r + 16 * k);
    }
    const int64_t srow = it.lse_off + (int64_t)u.z * L + min(qrow, L - 1);
    st.lse2 = a.lse2[srow];
    st.dlt = a.delta[srow];
  }
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) st.acc[mb] = f32x16{};
  const float c = a.scale_log2;

  for (int t = 0; t < n_tiles; t += 2) {
    wait_all_loads();
    __syncthreads();
    if (t + 1 < n_tiles) {
      ldK.load(sK1, (t + 1) * C::BN, L);
      ldV.load(sV1, (t + 1) * C::BN, L);
    }
    if (t < wave_tiles) dq_tile<D>(st, sK0, sV0, t * C::BN, wq0, qrow, lane, c);
    if (t + 1 >= n_tiles) break;
    wait_all_loads();
    __syncthreads();
    if (t + 2 < n_tiles) {
      ldK.load(sK0, (t + 2) * C::BN, L);
      ldV.load(sV0, (t + 2) * C::BN, L);
    }
    if (t + 1 < wave_tiles) dq_tile<D>(st, sK1, sV1, (t + 1) * C::BN, wq0, qrow, lane, c);
  }

  if (qrow < L) {
    const int64_t obase = qhead + (int64_t)qrow * qs;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * mb + 8 * gq + 4 * h;
        f32x4 v4 = {st.acc[mb][4 * gq] * a.scale, st.acc[mb][4 * gq + 1] * a.scale,
                    st.acc[mb][4 * gq + 2] * a.scale, st.acc[mb][4 * gq + 3] * a.scale};
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
  static constexpr int BN = kBwdBN;          // keys per unit (4 waves x 32)
  static constexpr int BM = kBwdBM;          // query rows per inner step
  static constexpr int QT = BM * D;          // elements of one Q or dO tile
  static constexpr int KS = D / 16;
  static constexpr int MB = D / 32;
};

template <int D>
struct KvState {
  bf16x8 kf[D / 16];   // K^T (B operand of S = Q K^T: column = key, k = head_dim)
  f32x16 dk[D / 32];   // dK^T (row = head_dim, column = key)
  f32x16 dv[D / 32];   // dV^T
};

// One 32-row query tile against this wave's 32 keys:
//   S = Q K^T, dP = dO V^T            (C layout: a key per lane, query rows in registers)
//   P = exp2(c S - lse2), dS = P (dP - Delta)
//   dV^T += dO^T P, dK^T += Q^T dS     (dO^T, Q^T via transpose reads)
// sVw points at this wave's 32 V rows in LDS (B operand of dP).
template <int D>
__device__ __forceinline__ void kv_tile(KvState<D> &st, const bf16 *sQ, const bf16 *sG, const float *sLD,
                                        const bf16 *sVw, int m0, int key, int kbase, int L, int lane, float c) {
  constexpr int KS = D / 16, MB = D / 32;
  const int l32 = lane & 31, h = lane >> 5;
  f32x16 s = f32x16{}, p = f32x16{};
#pragma unroll
  for (int k = 0; k < KS; ++k) {
    const int o = tile_off<D>(l32, 16 * k + 8 * h);
    s = mfma32x32x16(*(const bf16x8 *)(sQ + o), st.kf[k], s);
    p = mfma32x32x16(*(const bf16x8 *)(sG + o), *(const bf16x8 *)(sVw + o), p);
  }
  const bool mask = (m0 < kbase + 31) || (m0 + kBwdBM > L);
  bf16x8 pb[2], db[2];
#pragma unroll
  for (int g4 = 0; g4 < 4; ++g4) {
    const int qq = 8 * g4 + 4 * h;             // tile-local query row of element 4*g4
    const f32x4 l4 = *(const f32x4 *)(sLD + qq);
    const f32x4 d4 = *(const f32x4 *)(sLD + kBwdBM + qq);
#pragma unroll
    for (int x = 0; x < 4; ++x) {
      const int i = 4 * g4 + x;
      float e = fast_exp2(s[i] * c - l4[x]);
      if (mask) {
        const int q = m0 + qq + x;
        if (q < key || q >= L) e = 0.f;
      }
      pb[i >> 3][i & 7] = (bf16)e;
      db[i >> 3][i & 7] = (bf16)(e * (p[i] - d4[x]));
    }
  }
#pragma unroll
  for (int kk = 0; kk < 2; ++kk)
#pragma unroll
    for (int md = 0; md < MB; ++md) {
      st.dv[md] = mfma32x32x16(lds_tr_operand<D>(sG, 16 * kk, 32 * md, lane), pb[kk], st.dv[md]);
      st.dk[md] = mfma32x32x16(lds_tr_operand<D>(sQ, 16 * kk, 32 * md, lane), db[kk], st.dk[md]);
    }
}

// Loader of one inner step: Q and dO rows of a query tile plus lse2 and Delta
// (lanes 0..31 of wave 0 fetch lse2, lanes 32..63 Delta, one 4-byte lds load).
template <int D>
__device__ __forceinline__ void kv_load(const TileLoader<D, kBwdBM> &ldQ, const TileLoader<D, kBwdBM> &ldG,
                                        const float *lse2_row, const float *dlt_row, bf16 *sQ, bf16 *sG,
                                        float *sLD, int m, int L, int wave, int lane) {
  ldQ.load(sQ, m, L);
  ldG.load(sG, m, L);
  if (wave == 0) {
    const int q = min(m + (lane & 31), L - 1);
    const float *src = (lane < 32 ? lse2_row : dlt_row) + q;
    __builtin_amdgcn_global_load_lds((const void *)src, (__attribute__((address_space(3))) void *)sLD, 4, 0, 0);
  }
}

template <int D, bool G_F32>
__global__ void __launch_bounds__(256, 1) bwd_dkdv_kernel(AttnArgs a) {
  using C = KvCfg<D>;
  __shared__ __attribute__((aligned(16))) bf16 sV[C::BN * D];     // this unit's V rows
  __shared__ __attribute__((aligned(16))) bf16 sQ0[C::QT];
  __shared__ __attribute__((aligned(16))) bf16 sG0[C::QT];
  __shared__ __attribute__((aligned(16))) bf16 sQ1[C::QT];
  __shared__ __attribute__((aligned(16))) bf16 sG1[C::QT];
  __shared__ __attribute__((aligned(16))) float sLD0[2 * C::BM];  // lse2 | Delta
  __shared__ __attribute__((aligned(16))) float sLD1[2 * C::BM];

  const int4 u = a.units[blockIdx.x];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int n0 = u.y * C::BN;
  const int i_lo = u.z & 0xffff, i_hi = u.z >> 16;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const int64_t kvhead = it.kv_off + (int64_t)u.w * D;

  const int kbase = n0 + wave * 32;           // first key of this wave
  const int key = kbase + l32;                // this lane's key (MFMA column)
  const int mt0 = n0 / C::BM;                     // first query tile touching the keys
  const int mt_n = (L + C::BM - 1) / C::BM - mt0; // query tiles per head
  const int n_iter = (i_hi - i_lo) * mt_n;

  {
    const TileLoader<D, C::BN> ldV((const bf16 *)a.v + kvhead, ks, wave, lane);
    ldV.load(sV, n0, L);
  }
  KvState<D> st;
  {
    const bf16 *kp = (const bf16 *)a.k + kvhead + (int64_t)min(key, L - 1) * ks + 8 * h;
#pragma unroll
    for (int k = 0; k < C::KS; ++k) st.kf[k] = *(const bf16x8 *)(kp + 16 * k);
  }
#pragma unroll
  for (int md = 0; md < C::MB; ++md) { st.dk[md] = f32x16{}; st.dv[md] = f32x16{}; }
  const float c = a.scale_log2;

  // iteration i covers query head i_lo + i / mt_n, query tile mt0 + i % mt_n
  const bf16 *sVw = sV + wave * 32 * D;
  const int mt_end = mt0 + mt_n;
  int hd = i_lo, mt = mt0;
  TileLoader<D, C::BM> ldQ((const bf16 *)a.q + it.q_off + (int64_t)hd * D, qs, wave, lane);
  TileLoader<D, C::BM> ldG((const bf16 *)a.dout + it.q_off + (int64_t)hd * D, qs, wave, lane);
  const float *lrow = a.lse2 + it.lse_off + (int64_t)hd * L;
  const float *drow = a.delta + it.lse_off + (int64_t)hd * L;
  if (n_iter > 0) kv_load<D>(ldQ, ldG, lrow, drow, sQ0, sG0, sLD0, mt * C::BM, L, wave, lane);

  for (int itr = 0; itr < n_iter; itr += 2) {
    // even step: buffers 0 hold (hd, mt); prefetch the next step into buffers 1
    int cur_m = mt * C::BM;
    if (++mt == mt_end) {
      mt = mt0;
      ++hd;
      ldQ.src = (const bf16 *)a.q + it.q_off + (int64_t)hd * D;
      ldG.src = (const bf16 *)a.dout + it.q_off + (int64_t)hd * D;
      lrow = a.lse2 + it.lse_off + (int64_t)hd * L;
      drow = a.delta + it.lse_off + (int64_t)hd * L;
    }
    wait_all_loads();
    __syncthreads();
    if (itr + 1 < n_iter) kv_load<D>(ldQ, ldG, lrow, drow, sQ1, sG1, sLD1, mt * C::BM, L, wave, lane);
    if (cur_m + C::BM - 1 >= kbase) kv_tile<D>(st, sQ0, sG0, sLD0, sVw, cur_m, key, kbase, L, lane, c);
    if (itr + 1 >= n_iter) break;
    // odd step: buffers 1 hold (hd, mt); prefetch into buffers 0
    cur_m = mt * C::BM;
    if (++mt == mt_end) {
      mt = mt0;
      ++hd;
      ldQ.src = (const bf16 *)a.q + it.q_off + (int64_t)hd * D;
      ldG.src = (const bf16 *)a.dout + it.q_off + (int64_t)hd * D;
      lrow = a.lse2 + it.lse_off + (int64_t)hd * L;
      drow = a.delta + it.lse_off + (int64_t)hd * L;
    }
    wait_all_loads();
    __syncthreads();
    if (itr + 2 < n_iter) kv_load<D>(ldQ, ldG, lrow, drow, sQ0, sG0, sLD0, mt * C::BM, L, wave, lane);
    if (cur_m + C::BM - 1 >= kbase) kv_tile<D>(st, sQ1, sG1, sLD1, sVw, cur_m, key, kbase, L, lane, c);
  }

  if (key < L) {
    const int64_t obase = kvhead + (int64_t)key * ks;
#pragma unroll
    for (int md = 0; md < C::MB; ++md)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * md + 8 * gq + 4 * h;
        f32x4 k4 = {st.dk[md][4 * gq] * a.scale, st.dk[md][4 * gq + 1] * a.scale,
                    st.dk[md][4 * gq + 2] * a.scale, st.dk[md][4 * gq + 3] * a.scale};
        f32x4 v4 = {st.dv[md][4 * gq], st.dv[md][4 * gq + 1], st.dv[md][4 * gq + 2], st.dv[md][4 * gq + 3]};
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
