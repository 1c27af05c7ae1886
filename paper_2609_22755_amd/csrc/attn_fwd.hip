// Causal varlen grouped-query attention forward for gfx950.
//
// What is computed (per item j, local query head i, KV head g; positions are
// item-relative): O = softmax(scale * Q K^T + causal mask) V and the natural
// log-sum-exp of each row, i.e. exact attention over each complete sequence
// (the paper's FlashAttention compute step; Background, Sequence Packing and
// Sequence Parallelism).
//
// Work unit: (item, query head, 128-row query tile); four waves, each owning
// 32 query rows.  The wave computes S^T = K Q^T so that each lane owns one
// query row (the MFMA column) -- softmax statistics then live in a lane and
// need a single exchange between the two lane halves -- and O^T = V^T P^T,
// whose B operand is P^T straight from the S^T accumulator, and whose A
// operand V^T is read from the row-major LDS tile with ds_read_b64_tr_b16.
// Keys are processed 64 at a time, staged in LDS (row pitch D+16 elements),
// with the next tile's global loads in flight during the current tile's
// math.  Causality: tiles wholly above a wave's rows are skipped, and only
// tiles that straddle the diagonal evaluate the mask.
#include "device_common.hpp"
#include "nsp_internal.hpp"

namespace nsp {
namespace {

template <int D>
struct FwdCfg {
  static constexpr int BM = kFwdBM;
  static constexpr int BN = kFwdBN;
  static constexpr int LD = D + 16;          // LDS row pitch (elements)
  static constexpr int KS = D / 16;          // MFMA k-steps over head_dim
  static constexpr int MB = D / 32;          // 32-wide head_dim blocks
  static constexpr int CPR = D / 8;          // 16-byte chunks per row
  static constexpr int CPT = BN * CPR / 256; // chunks per thread per tile
};

template <int D, bool O_F32>
__global__ void __launch_bounds__(256) attn_fwd_kernel(AttnArgs a) {
  using C = FwdCfg<D>;
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
  const bf16 *Qh = (const bf16 *)a.q + it.q_off + (int64_t)u.z * D;
  const bf16 *Kg = (const bf16 *)a.k + it.kv_off + (int64_t)u.w * D;
  const bf16 *Vg = (const bf16 *)a.v + it.kv_off + (int64_t)u.w * D;

  const int wq0 = m0 + wave * 32;          // first query row of this wave
  const int qrow = wq0 + l32;              // this lane's query row
  const int qr = min(qrow, L - 1);

  // Q^T as the B operand of S^T = K Q^T: column = query row, k = head_dim.
  bf16x8 qf[C::KS];
#pragma unroll
  for (int s = 0; s < C::KS; ++s) qf[s] = *(const bf16x8 *)(Qh + qr * qs + 16 * s + 8 * h);

  f32x16 acc[C::MB];
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) acc[mb] = f32x16{};
  float m_run = -1e30f;   // running max of scale*log2(e)*S
  float l_run = 0.f;      // running sum of exp2(. - m_run)

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
    if (n0 > wq0 + 31) continue;   // every key of the tile is after every row of the wave

    // S^T for keys [n0, n0+64): two 32-key blocks.
    f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int st = 0; st < C::KS; ++st) {
        bf16x8 ak = *(const bf16x8 *)(sK + (kb * 32 + l32) * C::LD + 16 * st + 8 * h);
        s[kb] = mfma32x32x16(ak, qf[st], s[kb]);
      }
    }
    if (n0 + C::BN - 1 > wq0) {   // tile straddles this wave's diagonal
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = n0 + kb * 32 + 8 * (i >> 2) + 4 * h + (i & 3);
          if (key > qrow) s[kb][i] = -INFINITY;
        }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) mx = fmaxf(mx, s[kb][i]);
    mx = wave_max_halves(mx);
    const float m_new = fmaxf(m_run, mx * a.scale_log2);
    const float alpha = fast_exp2(m_run - m_new);
    float rs = 0.f;
    bf16x8 pb[4];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = fast_exp2(s[kb][i] * a.scale_log2 - m_new);
        rs += p;
        pb[kb * 2 + (i >> 3)][i & 7] = (bf16)p;
      }
    rs = wave_sum_halves(rs);
    l_run = l_run * alpha + rs;
    m_run = m_new;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb) acc[mb] *= alpha;

    // O^T += V^T P^T
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        bf16x8 av = lds_tr_operand(sV, C::LD, 16 * kk, 32 * mb, lane);
        acc[mb] = mfma32x32x16(av, pb[kk], acc[mb]);
      }
  }

  if (qrow < L) {
    const float inv = 1.f / l_run;
    const int64_t obase = it.q_off + (int64_t)qrow * qs + (int64_t)u.z * D;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * mb + 8 * gq + 4 * h;
        f32x4 v4 = {acc[mb][4 * gq] * inv, acc[mb][4 * gq + 1] * inv, acc[mb][4 * gq + 2] * inv,
                    acc[mb][4 * gq + 3] * inv};
        if constexpr (O_F32) {
          *(f32x4 *)((float *)a.o_out + obase + d0) = v4;
        } else {
          bf16x4 b4 = {(bf16)v4[0], (bf16)v4[1], (bf16)v4[2], (bf16)v4[3]};
          *(bf16x4 *)((bf16 *)a.o_out + obase + d0) = b4;
        }
      }
    if (h == 0) a.lse[it.lse_off + (int64_t)u.z * L + qrow] = (m_run + __log2f(l_run)) * kLn2;
  }
}

}  // namespace

hipError_t launch_attn_fwd(int head_dim, bool o_f32, const AttnArgs &a, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  dim3 grid(n_units), block(256);
  if (head_dim == 128) {
    if (o_f32) attn_fwd_kernel<128, true><<<grid, block, 0, s>>>(a);
    else attn_fwd_kernel<128, false><<<grid, block, 0, s>>>(a);
  } else {
    if (o_f32) attn_fwd_kernel<64, true><<<grid, block, 0, s>>>(a);
    else attn_fwd_kernel<64, false><<<grid, block, 0, s>>>(a);
  }
  return hipGetLastError();
}

}  // namespace nsp
