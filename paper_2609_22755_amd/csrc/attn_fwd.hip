// Causal varlen grouped-query attention forward for gfx950.
//
// What is computed (per item j, local query head i, KV head g; positions are
// item-relative): O = softmax(scale * Q K^T + causal mask) V and the natural
// log-sum-exp of each row, i.e. exact attention over each complete sequence
// (the paper's FlashAttention compute step; Background, Sequence Packing and
// Sequence Parallelism).
//
// Work unit: (item, query head, 256-row query tile); eight waves (two per
// SIMD), each owning 32 query rows.  The wave computes S^T = K Q^T so that
// each lane owns one query row (the MFMA column) -- softmax statistics then
// live in a lane and need a single exchange between the two lane halves -- and
// O^T = V^T P^T, whose B operand is P^T straight from the S^T accumulator, and
// whose A operand V^T is read from the row-major LDS tile with
// ds_read_b64_tr_b16 (LDS tiles use an XOR swizzle of 16-byte chunks against
// bank conflicts).  Keys are processed 64 at a time.  K and V tiles stream
// through a four-stage LDS ring filled by direct buffer->LDS loads
// (buffer_load_dwordx4 ... lds) issued three tiles ahead, with one barrier
// per tile; the 256 rows of a unit share every tile.  The accumulator is
// rescaled only when a row maximum grows by more than 2^8.  Causality: tiles
// wholly above a wave's rows are skipped, and only tiles that straddle the
// diagonal evaluate the mask.
#include "device_common.hpp"
#include "nsp_internal.hpp"

namespace nsp {
namespace {

template <int D>
struct FwdCfg {
  static constexpr int BM = kFwdBM;
  static constexpr int BN = kFwdBN;
  static constexpr int NW = kFwdWaves;
  static constexpr int TILE = BN * D;        // elements of one K or V tile (unpadded rows)
  static constexpr int KS = D / 16;          // MFMA k-steps over head_dim
  static constexpr int MB = D / 32;          // 32-wide head_dim blocks
  // buffer->LDS loads per wave and tile (K and V)
  static constexpr int LPW = 2 * TileLoader<D, BN, NW>::PER_WAVE;
  static_assert(BM == 32 * NW, "one 32-row block per wave");
};

// Rows whose running maximum grows by more than 2^kRescaleLog2 rescale the
// accumulator; otherwise the stale maximum is kept (exp2 values stay <= 2^8,
// exact in the final normalisation since the maximum cancels).
constexpr float kRescaleLog2 = 8.f;

// Per-wave state of the online softmax for 32 query rows.
template <int D>
struct FwdState {
  bf16x8 qf[D / 16];        // Q^T, B operand of S^T = K Q^T (column = query row, k = head_dim)
  f32x16 acc[D / 32];       // O^T (row = head_dim, column = query row)
  float m_run;              // reference maximum of scale*log2(e)*S (lazily updated)
  float l_run;              // sum of exp2(. - m_run)
};

// One 64-key tile: S^T = K Q^T, online softmax, O^T += V^T P^T.
template <int D>
__device__ __forceinline__ void fwd_tile(FwdState<D> &st, const bf16 *sK, const bf16 *sV, int n0, int wq0,
                                         int qrow, int lane, float c) {
  constexpr int KS = D / 16, MB = D / 32;
  const int l32 = lane & 31, h = lane >> 5;
  // S^T products in a fixed order, each K row operand read PF products ahead
  constexpr int NS = 2 * KS, PF = 4;
  f32x16 s0 = f32x16{}, s1 = f32x16{};
  bf16x8 op[NS];
#pragma unroll
  for (int f = 0; f < PF; ++f) op[f] = lds_row8<D>(sK, 32 * (f & 1) + l32, 16 * (f >> 1) + 8 * h);
#pragma unroll
  for (int j = 0; j < NS; ++j) {
    if (j + PF < NS) op[j + PF] = lds_row8<D>(sK, 32 * ((j + PF) & 1) + l32, 16 * ((j + PF) >> 1) + 8 * h);
    if (j & 1) s1 = mfma32x32x16(op[j], st.qf[j >> 1], s1);
    else s0 = mfma32x32x16(op[j], st.qf[j >> 1], s0);
    __builtin_amdgcn_sched_barrier(0);
  }
  if (n0 + kFwdBN - 1 > wq0) {   // tile straddles this wave's diagonal
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int key = n0 + 8 * (i >> 2) + 4 * h + (i & 3);
      if (key > qrow) s0[i] = -INFINITY;
      if (key + 32 > qrow) s1[i] = -INFINITY;
    }
  }
  // row maximum: two chains of three-operand maxima (v_max3_f32)
  float mxa = fmaxf(s0[0], s1[0]), mxb = fmaxf(s0[1], s1[1]);
#pragma unroll
  for (int i = 2; i < 16; i += 2) {
    mxa = fmaxf(fmaxf(mxa, s0[i]), s1[i]);
    mxb = fmaxf(fmaxf(mxb, s0[i + 1]), s1[i + 1]);
  }
  float mx = wave_max_halves(fmaxf(mxa, mxb)) * c;
  if (__any(mx > st.m_run + kRescaleLog2)) {
    const float m_new = fmaxf(st.m_run, mx);
    const float alpha = fast_exp2(st.m_run - m_new);
    st.l_run *= alpha;
    st.m_run = m_new;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb) st.acc[mb] *= alpha;
  }
  float rs = 0.f;
  bf16x8 pb[4];
#pragma unroll
  for (int i = 0; i < 16; ++i) {
    const float p0 = fast_exp2(s0[i] * c - st.m_run);
    const float p1 = fast_exp2(s1[i] * c - st.m_run);
    rs += p0 + p1;
    pb[i >> 3][i & 7] = (bf16)p0;
    pb[2 + (i >> 3)][i & 7] = (bf16)p1;
  }
  st.l_run += wave_sum_halves(rs);
#pragma unroll
  for (int kk = 0; kk < 4; ++kk)
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
      st.acc[mb] = mfma32x32x16(lds_tr_operand<D>(sV, 16 * kk, 32 * mb, lane), pb[kk], st.acc[mb]);
}

template <int D, bool O_F32>
__global__ void __launch_bounds__(64 * kFwdWaves, 1) attn_fwd_kernel(AttnArgs a) {
  using C = FwdCfg<D>;
  // K and V tiles, a four-stage ring: K of stage s at smem + s*TILE, V at
  // smem + (4+s)*TILE (for D = 128 the four K tiles lie within 64 KiB, so one
  // address register per operand serves every stage through the instruction
  // offset).  The ring is filled by loads the compiler does not track; the
  // waits and barriers of the steps order them against the reads.
  __shared__ __attribute__((aligned(16))) bf16 smem[8 * C::TILE];

  const int4 u = a.units[blockIdx.x];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int m0 = u.y * C::BM;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const bf16 *Qh = (const bf16 *)a.q + it.q_off + (int64_t)u.z * D;
  const TileLoader<D, C::BN, C::NW> ldK((const bf16 *)a.k + it.kv_off + (int64_t)u.w * D, ks, wave, lane);
  const TileLoader<D, C::BN, C::NW> ldV((const bf16 *)a.v + it.kv_off + (int64_t)u.w * D, ks, wave, lane);

  const int wq0 = m0 + wave * 32;          // first query row of this wave
  const int qrow = wq0 + l32;              // this lane's query row
  const int n_end = min(L, m0 + C::BM);
  const int n_tiles = (n_end + C::BN - 1) / C::BN;
  // tiles with keys <= this wave's rows (none for a wave wholly past the item end)
  const int wave_tiles = wq0 < L ? min(n_tiles, (wq0 + 31) / C::BN + 1) : 0;

  FwdState<D> st;
  {
    const bf16 *qp = Qh + (int64_t)min(qrow, L - 1) * qs + 8 * h;
#pragma unroll
    for (int k = 0; k < C::KS; ++k) st.qf[k] = *(const bf16x8 *)(qp + 16 * k);
  }
  // The query-side registers land before the tile loads are issued: the
  // compiler does not count those loads, so a wait of its own for these
  // registers inside the loop would drain the ring.
  wait_all_loads();
  // tiles 0..2 in flight (past the item end a tile load fetches nothing)
  for (int j = 0; j < 3; ++j) {
    ldK.load_untracked(smem + j * C::TILE, j * C::BN, L);
    ldV.load_untracked(smem + (4 + j) * C::TILE, j * C::BN, L);
  }
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) st.acc[mb] = f32x16{};
  st.m_run = -INFINITY;
  st.l_run = 0.f;
  const float c = a.scale_log2;

  // step t: wait for this wave's loads of tile t (those of t+1, t+2 may stay
  // in flight), barrier (every wave's part of tile t has landed and every
  // wave is done with tile t-1), refill tile t-1's stage with tile t+3, and
  // process tile t.
  int t = 0;
  for (;;) {
#define NSP_FWD_STEP(CUR, FILL)                                                      \
    {                                                                               \
      wait_loads_le<2 * C::LPW>();                                                  \
      stage_barrier();                                                              \
      ldK.load_untracked(smem + (FILL) * C::TILE, (t + 3) * C::BN, L);              \
      ldV.load_untracked(smem + (4 + (FILL)) * C::TILE, (t + 3) * C::BN, L);        \
      if (t < wave_tiles)                                                           \
        fwd_tile<D>(st, smem + (CUR) * C::TILE, smem + (4 + (CUR)) * C::TILE, t * C::BN, wq0, qrow, lane, c); \
      if (++t >= n_tiles) break;                                                    \
    }
    NSP_FWD_STEP(0, 3)
    NSP_FWD_STEP(1, 0)
    NSP_FWD_STEP(2, 1)
    NSP_FWD_STEP(3, 2)
#undef NSP_FWD_STEP
  }
  // no buffer->LDS load may still be in flight when the workgroup ends
  wait_all_loads();

  if (qrow < L) {
    const float inv = 1.f / st.l_run;
    const int64_t obase = it.q_off + (int64_t)qrow * qs + (int64_t)u.z * D;
#pragma unroll
    for (int mb = 0; mb < C::MB; ++mb)
#pragma unroll
      for (int gq = 0; gq < 4; ++gq) {
        const int d0 = 32 * mb + 8 * gq + 4 * h;
        f32x4 v4 = {st.acc[mb][4 * gq] * inv, st.acc[mb][4 * gq + 1] * inv, st.acc[mb][4 * gq + 2] * inv,
                    st.acc[mb][4 * gq + 3] * inv};
        if constexpr (O_F32) {
          *(f32x4 *)((float *)a.o_out + obase + d0) = v4;
        } else {
          bf16x4 b4 = {(bf16)v4[0], (bf16)v4[1], (bf16)v4[2], (bf16)v4[3]};
          *(bf16x4 *)((bf16 *)a.o_out + obase + d0) = b4;
        }
      }
    if (h == 0) a.lse[it.lse_off + (int64_t)u.z * L + qrow] = (st.m_run + __log2f(st.l_run)) * kLn2;
  }
}

}  // namespace

hipError_t launch_attn_fwd(int head_dim, bool o_f32, const AttnArgs &a, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  dim3 grid(n_units), block(64 * kFwdWaves);
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
