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
// bank conflicts).  Keys are processed 64 at a time.  Each wave is software
// pipelined: the S^T products of tile t+1 and the PV products of tile t run
// on the matrix cores while the vector units compute P of tile t and the row
// maxima of tile t+1.  K and V tiles stream through two four-stage LDS rings
// (K one tile ahead of V) filled by direct buffer->LDS loads
// (buffer_load_dwordx4 ... lds) issued three steps ahead, with one barrier
// per step; the 256 rows of a unit share every tile.  The accumulator is
// rescaled only when a row maximum grows by more than 2^8.  Causality: tiles
// wholly above a wave's rows are skipped, and only tiles that straddle the
// diagonal evaluate the mask.
#include <algorithm>
#include <functional>
#include <mutex>
#include <unordered_map>
#include <utility>

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
  // the tiles are loaded by the first NL waves (one per SIMD): while a
  // loading wave waits for the memory pipeline to accept its loads, the other
  // wave on its SIMD keeps the matrix core busy
  static constexpr int NL = 4;
  // buffer->LDS loads per loading wave and tile (K and V)
  static constexpr int LPW = 2 * TileLoader<D, BN, NL>::PER_WAVE;
  static_assert(BM == 32 * NW, "one 32-row block per wave");
};

// Rows whose running maximum grows by more than 2^kRescaleLog2 rescale the
// accumulator; otherwise the stale maximum is kept (exp2 values stay <= 2^8,
// exact in the final normalisation since the maximum cancels).
constexpr float kRescaleLog2 = 8.f;

// LDS operand prefetch distance of the forward half-steps, in products.
constexpr int kFwdPf = 3;

// Per-wave state of the online softmax for 32 query rows.
template <int D>
struct FwdState {
  bf16x8 qf[D / 16];        // Q^T, B operand of S^T = K Q^T (column = query row, k = head_dim)
  f32x16 acc[D / 32];       // O^T (row = head_dim, column = query row)
  float m_run;              // reference maximum of scale*log2(e)*S (lazily updated)
  float l_part;             // this lane's part of the row sum of exp2(. - m_run)
  bf16x8 op0[kFwdPf];       // LDS operands of the next half-step's first products, read ahead
};

// LDS byte addresses of this lane's operand reads, relative to the start of
// a tile, computed once per kernel.  Every read adds a compile-time byte
// offset (ring stage, 32-key half, 16-key block) that the instruction's
// offset field absorbs, so the loop needs no address arithmetic and no
// per-stage address registers.  The values are hidden from the compiler
// (which would otherwise re-derive an address per stage and offset).
template <int D>
struct FwdAddr {
  unsigned k[D / 16];       // K row operand, k block k (rows l%32, keys of a half)
  unsigned v[D / 32][2];    // V^T transpose reads, head_dim block mb, rows 0..7 / 8..15 of a 16-key block
  __device__ __forceinline__ FwdAddr(int lane, unsigned k_ring) {
    const int l32 = lane & 31, h = lane >> 5, g = lane >> 4, j = lane & 15;
#pragma unroll
    for (int kb = 0; kb < D / 16; ++kb) {
      k[kb] = k_ring + 2u * (unsigned)tile_off<D>(l32, 16 * kb + 8 * h);
      asm volatile("" : "+v"(k[kb]));
    }
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int hi = 0; hi < 2; ++hi) {
        v[mb][hi] = 2u * (unsigned)tile_off<D>(4 * h + (j >> 2) + 8 * hi, 32 * mb + 16 * (g & 1) + 4 * (j & 3));
        asm volatile("" : "+v"(v[mb][hi]));
      }
  }
};

__device__ __forceinline__ bf16x8 lds_b128_at(const bf16 *lds, unsigned byte_addr) {
  return *(const bf16x8 *)((const char *)lds + byte_addr);
}
__device__ __forceinline__ bf16x4 lds_tr4_at(const bf16 *lds, unsigned byte_addr) {
  return lds_read_tr4((const bf16 *)((const char *)lds + byte_addr));
}

// LDS operand of product f of a half-step: f < KS: K row operand of
// S^T = K Q^T for the next 32 keys (k block f, tile rows from kn_off); then
// the 2*MB products of O^T += V^T P^T for the current 32 keys (k block
// kk = g/MB of 16 keys, head_dim block mb = g%MB, g = f - KS, tile rows from
// v_off), V^T by transpose reads.  kn_off / v_off are byte offsets (ring
// stage + row offset; row offsets are multiples of 16, which the swizzle does
// not see).
template <int D>
__device__ __forceinline__ bf16x8 fwd_operand(int f, const bf16 *smem, const FwdAddr<D> &ad, unsigned kn_off,
                                              unsigned v_off) {
  constexpr int KS = D / 16, MB = D / 32;
  if (f < KS) return lds_b128_at(smem, ad.k[f] + kn_off);
  const int g = f - KS;
  const unsigned o = v_off + 2u * 16u * D * (unsigned)(g / MB);
  return cat4(lds_tr4_at(smem, ad.v[g % MB][0] + o), lds_tr4_at(smem, ad.v[g % MB][1] + o));
}

// Set the scores of keys past this lane's query row to -inf: the wave's
// diagonal half (keys n0..n0+31 against rows n0..n0+31).
__device__ __forceinline__ void fwd_mask(f32x16 &s, int n0, int qrow, int h) {
#pragma unroll
  for (int i = 0; i < 16; ++i)
    if (n0 + 8 * (i >> 2) + 4 * h + (i & 3) > qrow) s[i] = -INFINITY;
}

// One half-step over 32 keys, software pipelined within the wave:
//   * on entry `sc` holds the (masked) scores S^T of these keys and st.m_run
//     already covers their row maxima;
//   * the matrix cores compute S^T of the next 32 keys into `sn`, then
//     O^T += V^T P^T of these keys;
//   * beside those products the vector units turn these keys into
//     P = exp2(c S - m_run) (packed to bf16 for the PV products, summed in
//     float32) and take the row maxima of the next keys.
// The products run as a fixed sequence of chunks, each issuing the LDS
// operand PF products ahead (the last chunks read the first operands of the
// next half-step, K rows at kn_next, into st.op0, so that no half-step
// starts by waiting for its operands), with about four vector instructions
// beside each product; a scheduling fence after each chunk keeps that order, and each
// vector result is pinned to its chunk (pin()), since the compiler would
// otherwise sink the ones without consumers in the chunk to the end.  The
// wave's last half-step computes next scores too (from LDS rows that are
// never used) so that every half-step runs the same code; its caller discards
// them.  Returns the unmasked row maximum (scaled, base 2) of the next keys.
template <int D>
__device__ __forceinline__ float fwd_half(FwdState<D> &st, f32x16 &sc, f32x16 &sn, const bf16 *smem,
                                          const FwdAddr<D> &ad, unsigned kn_off, unsigned v_off, unsigned kn_next,
                                          float c) {
  constexpr int KS = D / 16, MB = D / 32;
  constexpr int NS = KS;                       // S^T products of the next keys
  constexpr int NP = NS + 2 * MB;              // products in this half-step
  constexpr int PF = kFwdPf;
  static_assert(PF <= KS, "the read-ahead operands are K rows");
  // chunk of the first vector op of score element e: spread so that the bf16
  // group of keys 16kk.. is packed before the PV products of k block kk start
  // (chunk NS + MB*kk); the float32 row-sum additions come later, from chunk
  // NS + MB - 1 on
  constexpr int F = NS + MB - 3;
  constexpr int A0 = NS + MB - 1;
  bf16x8 op[NP + PF];
  bf16x8 pb[2];
  float mxa = -INFINITY, mxb = -INFINITY;
  float rs0 = 0.f, rs1 = 0.f;
  sn = f32x16{};
#pragma unroll
  for (int f = 0; f < PF; ++f) op[f] = st.op0[f];
#pragma clang loop unroll(full)
  for (int pj = 0; pj < NP; ++pj) {
    if (pj + PF < NP) op[pj + PF] = fwd_operand<D>(pj + PF, smem, ad, kn_off, v_off);
    else op[pj + PF] = fwd_operand<D>(pj + PF - NP, smem, ad, kn_next, 0);
    if (pj < NS) {
      sn = mfma32x32x16(op[pj], st.qf[pj], sn);
    } else {
      const int g = pj - NS;
      st.acc[g % MB] = mfma32x32x16(op[pj], pb[g / MB], st.acc[g % MB]);
    }
    // P of these keys: scale-and-shift, exp2, then pack by pairs; sums later
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int fe = e * F / 16;
      if (pj == fe) sc[e] = pin(sc[e] * c - st.m_run);
      if (pj == fe + 1) sc[e] = pin(fast_exp2(sc[e]));
      if ((e & 1) && pj == fe + 2) {
        pb[e >> 3][(e & 7) - 1] = (bf16)sc[e - 1];
        pb[e >> 3][e & 7] = (bf16)sc[e];
      }
      if (pj == A0 + e * (NP - A0) / 16) {
        if (e & 1) rs1 = pin(rs1 + sc[e]);
        else rs0 = pin(rs0 + sc[e]);
      }
    }
    // row maxima of the next keys, two chains of three-operand maxima
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (pj == NS + 2 + i * (2 * MB - 3) / 4) {
        mxa = pin(fmaxf(fmaxf(mxa, sn[4 * i]), sn[4 * i + 1]));
        mxb = pin(fmaxf(fmaxf(mxb, sn[4 * i + 2]), sn[4 * i + 3]));
      }
    __builtin_amdgcn_sched_barrier(0);
  }
  st.l_part += rs0 + rs1;
#pragma unroll
  for (int f = 0; f < PF; ++f) st.op0[f] = op[NP + f];
  return wave_max_halves(fmaxf(mxa, mxb)) * c;
}

// Raise the reference maximum to cover `mx` (the scaled maxima of the keys
// about to be exponentiated) when it grew by more than 2^kRescaleLog2, and
// rescale the accumulator and row sum to match.
template <int D>
__device__ __forceinline__ void fwd_update_max(FwdState<D> &st, float mx) {
  if (__any(mx > st.m_run + kRescaleLog2)) {
    const float m_new = fmaxf(st.m_run, mx);
    const float alpha = fast_exp2(st.m_run - m_new);
    st.l_part *= alpha;
    st.m_run = m_new;
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb) st.acc[mb] *= alpha;
  }
}

// Scaled (base 2) row maximum of a block of scores.
__device__ __forceinline__ float fwd_block_max(const f32x16 &s, float c) {
  float mx = fmaxf(s[0], s[1]);
#pragma unroll
  for (int i = 2; i < 16; i += 2) mx = fmaxf(fmaxf(mx, s[i]), s[i + 1]);
  return wave_max_halves(mx) * c;
}

// Half-step u (keys 32u .. 32u+31) of a wave that processes `halves` halves;
// waves already done skip it.  The last one, u = halves-1, is the wave's
// diagonal block: it masks its scores and updates the reference maximum from
// the masked ones first (the half-step before it computes these scores but
// leaves the maximum alone, so that keys past a row never raise it).
template <int D>
__device__ __forceinline__ void fwd_half_step(FwdState<D> &st, f32x16 &sc, f32x16 &sn, const bf16 *smem,
                                              const FwdAddr<D> &ad, unsigned kn_off, unsigned v_off,
                                              unsigned kn_next, int u, int halves, int qrow, int h, float c) {
  if (u < halves) {
    if (u + 1 == halves) {
      fwd_mask(sc, 32 * u, qrow, h);
      fwd_update_max<D>(st, fwd_block_max(sc, c));
    }
    const float mx = fwd_half<D>(st, sc, sn, smem, ad, kn_off, v_off, kn_next, c);
    if (u + 2 < halves) fwd_update_max<D>(st, mx);
  }
}

// One forward unit (launch slot `slot` of the unit list).  smem: K and V
// tiles, two four-stage rings: V tile t in stage t%4 at smem + (t%4)*TILE, K
// tile t at smem + (4 + t%4)*TILE.  Each ring spans at most 64 KiB, so every
// read is one of the per-lane addresses of FwdAddr plus an instruction
// offset.  Step t reads K of tiles t and t+1 and V of tile t.  The rings are
// filled by loads the compiler does not track; the waits and barriers of the
// steps order them against the reads.
template <int D, bool O_F32>
__device__ __forceinline__ void fwd_unit(const AttnArgs &a, int slot, bf16 *smem) {
  using C = FwdCfg<D>;
  const int4 u = a.units[slot];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int m0 = u.y * C::BM;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const bf16 *Qh = (const bf16 *)a.q + it.q_off + (int64_t)u.z * D;
  const bool loader = wave < C::NL;
  const TileLoader<D, C::BN, C::NL> ldK((const bf16 *)a.k + it.kv_off + (int64_t)u.w * D, ks, wave % C::NL, lane);
  const TileLoader<D, C::BN, C::NL> ldV((const bf16 *)a.v + it.kv_off + (int64_t)u.w * D, ks, wave % C::NL, lane);

  const int wq0 = m0 + wave * 32;          // first query row of this wave
  const int qrow = wq0 + l32;              // this lane's query row
  const int n_end = min(L, m0 + C::BM);
  const int n_tiles = (n_end + C::BN - 1) / C::BN;
  // 32-key halves with keys <= this wave's rows: the last one is the wave's
  // diagonal block (none for a wave wholly past the item end)
  const int halves = wq0 < L ? wq0 / 32 + 1 : 0;

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
  if (loader)
    for (int j = 0; j < 3; ++j) {
      ldK.load_untracked(smem + (4 + j) * C::TILE, j * C::BN, L);
      ldV.load_untracked(smem + j * C::TILE, j * C::BN, L);
    }
  const FwdAddr<D> ad(lane, 2u * 4u * C::TILE);
  constexpr unsigned TB = 2u * C::TILE;       // bytes per tile
  constexpr unsigned HB = 2u * 32u * D;       // bytes per 32 rows
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) st.acc[mb] = f32x16{};
  st.m_run = -INFINITY;
  st.l_part = 0.f;
  const float c = a.scale_log2;

  // scores of keys 0..31 (every wave with rows in the item has keys there)
  f32x16 sa, sb;
  wait_loads_le<2 * C::LPW>();
  stage_barrier();
  if (halves > 0) {
    sa = f32x16{};
#pragma unroll
    for (int k = 0; k < C::KS; ++k) sa = mfma32x32x16(lds_b128_at(smem, ad.k[k]), st.qf[k], sa);
    // (keys 0..31 are the diagonal block of wave 0: its first half-step
    // takes their maximum after masking)
    if (halves > 1) fwd_update_max<D>(st, fwd_block_max(sa, c));
    // the first operands of the first half-step (K tile 0, rows 32..63)
#pragma unroll
    for (int f = 0; f < kFwdPf; ++f) st.op0[f] = fwd_operand<D>(f, smem, ad, HB, 0);
  }

  // step t: wait for this wave's loads of tile t+1 (those of tile t+2 may
  // stay in flight), barrier (every wave's part has landed and every wave is
  // done with step t-1), refill stage (t-1)%4 with tile t+3, then two
  // half-steps: keys 64t.. (next scores from K tile t, rows 32..63) and keys
  // 64t+32.. (next scores from K tile t+1, rows 0..31).
  int t = 0;
  for (;;) {
#define NSP_FWD_STEP(CUR)                                                                   \
    {                                                                                      \
      wait_loads_le<C::LPW>();                                                             \
      stage_barrier();                                                                     \
      if (loader) {                                                                        \
        ldK.load_untracked(smem + (4 + (((CUR) + 3) & 3)) * C::TILE, (t + 3) * C::BN, L);  \
        ldV.load_untracked(smem + (((CUR) + 3) & 3) * C::TILE, (t + 3) * C::BN, L);        \
      }                                                                                    \
      fwd_half_step<D>(st, sa, sb, smem, ad, (CUR) * TB + HB, (CUR) * TB, (((CUR) + 1) & 3) * TB, 2 * t,   \
                       halves, qrow, h, c);                                                \
      fwd_half_step<D>(st, sb, sa, smem, ad, (((CUR) + 1) & 3) * TB, (CUR) * TB + HB,                    \
                       (((CUR) + 1) & 3) * TB + HB, 2 * t + 1, halves, qrow, h, c);                 \
      if (++t >= n_tiles) break;                                                           \
    }
    NSP_FWD_STEP(0)
    NSP_FWD_STEP(1)
    NSP_FWD_STEP(2)
    NSP_FWD_STEP(3)
#undef NSP_FWD_STEP
  }
  // no buffer->LDS load may still be in flight when the workgroup ends
  wait_all_loads();

  const float l_run = wave_sum_halves(st.l_part);
  if (qrow < L) {
    const float inv = 1.f / l_run;
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
    if (h == 0) a.lse[it.lse_off + (int64_t)u.z * L + qrow] = (st.m_run + __log2f(l_run)) * kLn2;
  }
}

// The forward pass.  With queue heads (a.queue: kXcdQueues heads and a
// count of workgroups done, zero at launch), one persistent workgroup per
// compute unit takes units from the per-XCD queues, and the last workgroup
// to finish sets them back to zero for the next launch on the same stream.
// Without (a.queue == nullptr), workgroup b runs launch slot b.
template <int D, bool O_F32>
__global__ void __launch_bounds__(64 * kFwdWaves, 1) attn_fwd_kernel(AttnArgs a, int n_units) {
  __shared__ __attribute__((aligned(16))) bf16 smem[8 * FwdCfg<D>::TILE];
  __shared__ int s_slot;
  const int own = (int)(__builtin_amdgcn_s_getreg(kHwRegXccId) % kXcdQueues);
  for (int iter = 0;; ++iter) {
    const int slot = a.queue ? next_queue_slot(a.queue, n_units, own, &s_slot) : (iter == 0 ? (int)blockIdx.x : -1);
    if (slot < 0) break;
    fwd_unit<D, O_F32>(a, slot, smem);
  }
  // every fetch of this workgroup has returned before its count is added
  // (thread 0 made both, the fetch's result decided to stop), so the last
  // workgroup counted knows that no fetch of this launch is still to come
  if (a.queue && threadIdx.x == 0 && atomicAdd(a.queue + kXcdQueues, 1) == (int)gridDim.x - 1) {
    for (int x = 0; x < kXcdQueues; ++x) atomicExch(a.queue + x, 0);
    atomicExch(a.queue + kXcdQueues, 0);
  }
}

// Zero the queue heads of a counter block (run once, when the block is
// first given to a stream).
__global__ void zero_ints_kernel(int *p, int n) {
  if ((int)threadIdx.x < n) p[threadIdx.x] = 0;
}

// Counter blocks of the persistent forward, one per (device, stream) that
// has launched it: kXcdQueues heads and a done count each, padded to 64
// bytes.  The array lives with the module on every device; host code uses
// each device's address of it (looked up once per device).  Calls on one
// stream run one after another, so they can share a block; calls on
// different streams get different blocks.
constexpr int kFwdBlockInts = 16;
constexpr int kFwdBlocks = 4096;
__device__ __align__(256) int fwd_queue_blocks[kFwdBlocks * kFwdBlockInts];

struct DevStream {
  int dev;
  hipStream_t stream;
  bool operator==(const DevStream &o) const { return dev == o.dev && stream == o.stream; }
};
struct DevStreamHash {
  size_t operator()(const DevStream &k) const {
    return std::hash<const void *>()((const void *)k.stream) * 31u + (size_t)k.dev;
  }
};
std::mutex g_fwd_mu;
std::unordered_map<int, std::pair<int *, int>> g_fwd_dev;            // device -> (array address, blocks given)
std::unordered_map<DevStream, int *, DevStreamHash> g_fwd_block;     // (device, stream) -> its block

// The counter block of `s` on the current device (nullptr once every block
// has been given out: the caller then launches one workgroup per unit).
hipError_t fwd_queue_block(hipStream_t s, int **out) {
  *out = nullptr;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  std::lock_guard<std::mutex> lock(g_fwd_mu);
  auto it = g_fwd_block.find(DevStream{dev, s});
  if (it != g_fwd_block.end()) {
    *out = it->second;
    return hipSuccess;
  }
  auto d = g_fwd_dev.find(dev);
  if (d == g_fwd_dev.end()) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(fwd_queue_blocks));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    d = g_fwd_dev.emplace(dev, std::make_pair(static_cast<int *>(p), 0)).first;
  }
  if (d->second.second >= kFwdBlocks) return hipSuccess;
  int *blk = d->second.first + (size_t)kFwdBlockInts * d->second.second;
  zero_ints_kernel<<<1, kFwdBlockInts, 0, s>>>(blk, kFwdBlockInts);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  ++d->second.second;
  g_fwd_block.emplace(DevStream{dev, s}, blk);
  *out = blk;
  return hipSuccess;
}


}  // namespace

hipError_t launch_attn_fwd(int head_dim, bool o_f32, const AttnArgs &a_in, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  AttnArgs a = a_in;
  a.queue = nullptr;
  int cus = 0;
  hipError_t e = compute_units(&cus);
  if (e != hipSuccess) return e;
  // with more units than compute units, one persistent workgroup per compute
  // unit (its resources allow no more) on the stream's counter block;
  // otherwise, or without a block, one workgroup per unit
  if (n_units > cus) {
    e = fwd_queue_block(s, &a.queue);
    if (e != hipSuccess) return e;
  }
  dim3 grid(a.queue ? cus : n_units), block(64 * kFwdWaves);
  if (head_dim == 128) {
    if (o_f32) attn_fwd_kernel<128, true><<<grid, block, 0, s>>>(a, n_units);
    else attn_fwd_kernel<128, false><<<grid, block, 0, s>>>(a, n_units);
  } else {
    if (o_f32) attn_fwd_kernel<64, true><<<grid, block, 0, s>>>(a, n_units);
    else attn_fwd_kernel<64, false><<<grid, block, 0, s>>>(a, n_units);
  }
  return hipGetLastError();
}

}  // namespace nsp
