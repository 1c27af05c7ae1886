// Causal varlen grouped-query attention backward for gfx950.
//
// The analytic gradient of the forward (exact attention per sequence):
//   P = exp(scale*S - lse), Delta[t] = <dO[t], O[t]>, dP = dO V^T,
//   dS = P * (dP - Delta), dQ = scale * dS K, dK = scale * dS^T Q, dV = P^T dO,
// with dK/dV summed over the local query heads that share a KV head.
//
// Three passes, deterministic (no atomics; every output element is written
// by exactly one lane):
//   preprocess : -Delta per (item, head, row) and lse*log2(e), float32,
//                layout of lse (-Delta starts the dP product chains).
//   dK/dV      : unit = (item, KV head, 128-key tile); four waves, each owning
//                32 keys whose K and V rows stay in registers.  The unit loops
//                over the 64-row query tiles at or past its diagonal -- up
//                from the diagonal, or down from the item end for a unit so
//                flagged -- and, per tile, over the query heads of the KV
//                head's group (the host pairs and orders the units so that
//                the units running at once on one XCD read the same tiles at
//                the same time, see the schedule builder); each tile's
//                Q, dO, lse2 and Delta stream into a four-stage LDS ring with
//                direct buffer->LDS loads issued three tiles ahead, one per
//                product in the first products of a step.  S = Q K^T
//                puts a key in each lane, so P and dS (C layout) feed
//                dV^T = dO^T P and dK^T = Q^T dS as B operands; dO^T and Q^T
//                are read from the row-major tiles with ds_read_b64_tr_b16.
//                A tile is taken in two 32-row sub-steps, software pipelined
//                for one wave per SIMD: the S / dP products of sub-tile j+1
//                run on the matrix cores while the vector units compute P
//                and dS of sub-tile j, in a fixed instruction order.
//   dQ         : unit = (item, query head, 256-row tile), like the forward:
//                S^T = K Q^T and dP^T = V dO^T put a query row in each lane;
//                dQ^T = K^T dS^T takes dS^T as B operand and K^T from the
//                row-major K tile via transpose reads; K and V tiles stream
//                through a four-stage LDS ring, loaded three tiles ahead.
#include <algorithm>

#include "device_common.hpp"
#include "nsp_internal.hpp"

namespace nsp {
namespace {

constexpr int kQueueSlots = 64;  // queue-head ints the preprocess resets (the workspace holds 256 bytes)
constexpr int kKvQueue0 = 0;     // heads of the dK/dV pass's queues: slots 0..7
constexpr int kDqQueue0 = 8;     // heads of the dQ pass's queues: slots 8..15

// ------------------------------------------------------------ preprocess --

// -Delta[t] = -sum_d dO[t,i,d] * O[t,i,d], and lse2 = lse * log2(e) (the
// backward works in base 2).  Workgroup b covers the tokens of
// a.pre_blocks[b] for one local query head (only the items the call computes
// have blocks): one group of D/8 lanes per token, U tokens per lane group in
// flight; consecutive lane groups take consecutive tokens, so that their
// LSE / Delta entries are adjacent.  Block 0 also resets the unit-queue heads
// that the passes after it on the same stream take their units from (a call
// with no rows to process has no units either).
template <int D, bool O_F32>
__global__ void __launch_bounds__(256) bwd_preprocess_kernel(AttnArgs a) {
  if (blockIdx.x == 0 && threadIdx.x < kQueueSlots) a.queue[threadIdx.x] = 0;
  constexpr int LPR = D / 8;                 // lanes per token
  constexpr int TPP = 256 / LPR;             // tokens per pass of the workgroup
  constexpr int U = 4;                       // passes in flight
  const PreBlock pb = a.pre_blocks[blockIdx.x];
  const ItemDesc it = a.items[pb.item];
  const int sub = threadIdx.x % LPR;
  const int tl = threadIdx.x / LPR;
  const int64_t row_stride = (int64_t)it.hq * D;            // elements between tokens
  const int64_t head_base = it.q_off + (int64_t)pb.head * D + sub * 8;
  const int64_t lse_base = it.lse_off + (int64_t)pb.head * it.L;
  for (int base = 0; base < pb.ntok; base += TPP * U) {
    float acc[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      acc[u] = 0.f;
      const int k = base + u * TPP + tl;
      if (k < pb.ntok) {
        const int64_t e = head_base + (int64_t)(pb.t0 + k) * row_stride;
        const bf16x8 g = *(const bf16x8 *)((const bf16 *)a.dout + e);
        if constexpr (O_F32) {
          const f32x4 o0 = *(const f32x4 *)((const float *)a.o + e);
          const f32x4 o1 = *(const f32x4 *)((const float *)a.o + e + 4);
#pragma unroll
          for (int x = 0; x < 4; ++x) acc[u] += (float)g[x] * o0[x] + (float)g[x + 4] * o1[x];
        } else {
          const bf16x8 o = *(const bf16x8 *)((const bf16 *)a.o + e);
#pragma unroll
          for (int x = 0; x < 8; ++x) acc[u] += (float)g[x] * (float)o[x];
        }
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int off = LPR / 2; off >= 1; off >>= 1) acc[u] += __shfl_xor(acc[u], off);
      const int k = base + u * TPP + tl;
      if (k < pb.ntok && sub == 0) {
        const int64_t o = lse_base + pb.t0 + k;
        a.delta[o] = -acc[u];      // stored negated: the start of the dP product chains
        a.lse2[o] = a.lse_in[o] * kLog2e;
      }
    }
  }
}

// -------------------------------------------------------------------- dQ --

template <int D>
struct DqCfg {
  static constexpr int BM = kFwdBM;
  static constexpr int BN = kFwdBN;
  static constexpr int NW = kFwdWaves;
  static constexpr int TILE = BN * D;
  static constexpr int KS = D / 16;
  static constexpr int MB = D / 32;
  // the tiles are loaded by the first NL waves (one per SIMD), as in the
  // forward
  static constexpr int NL = 4;
  static constexpr int LPW = 2 * TileLoader<D, BN, NL>::PER_WAVE;   // loads per loading wave and tile
};

template <int D>
struct DqState {
  bf16x8 qf[D / 16];   // Q^T  (B operand: column = query row, k = head_dim)
  bf16x8 gf[D / 16];   // dO^T (B operand)
  f32x16 acc[D / 32];  // dQ^T (row = head_dim, column = query row)
  f32x16 ndlt;         // -Delta of the lane's query row in every element: the
                       // starting value of each dP^T product chain, which
                       // then ends at dP^T - Delta
  float lse2;
};

// Per-lane LDS byte addresses of the dQ kernel's operand reads within a ring
// stage (computed once, hidden from the compiler; every read adds the stage,
// half and block offsets through the instruction's offset field).
template <int D>
struct DqAddr {
  unsigned kr[D / 16];      // K row operand of a 32-key half, k block k (K ring)
  unsigned vr[D / 16];      // the same in the V ring
  unsigned kt[D / 32][2];   // K^T transpose reads, head_dim block mb, rows 0..7 / 8..15
  __device__ __forceinline__ DqAddr(int lane, unsigned v_ring) {
    const int l32 = lane & 31, h = lane >> 5, g = lane >> 4, j = lane & 15;
#pragma unroll
    for (int k = 0; k < D / 16; ++k) {
      kr[k] = 2u * (unsigned)tile_off<D>(l32, 16 * k + 8 * h);
      vr[k] = v_ring + kr[k];
      asm volatile("" : "+v"(kr[k]));
      asm volatile("" : "+v"(vr[k]));
    }
#pragma unroll
    for (int mb = 0; mb < D / 32; ++mb)
#pragma unroll
      for (int hi = 0; hi < 2; ++hi) {
        kt[mb][hi] = 2u * (unsigned)tile_off<D>(4 * h + (j >> 2) + 8 * hi, 32 * mb + 16 * (g & 1) + 4 * (j & 3));
        asm volatile("" : "+v"(kt[mb][hi]));
      }
  }
};

// LDS operand of product f of a 64-key tile: per 32-key half kb (f in
// [NH*kb, NH*kb + NH), NH = 2*KS + 2*MB): first the rows of K (even) and V
// (odd) for S^T = K Q^T and dP^T = V dO^T, k block (f%NH)/2; then the
// transposed K for dQ^T += K^T dS^T, k block kk = g/MB and head_dim block
// md = g%MB, g = f%NH - 2*KS.
template <int D>
__device__ __forceinline__ bf16x8 dq_operand(int f, const bf16 *smem, const DqAddr<D> &ad, unsigned so) {
  using C = DqCfg<D>;
  constexpr int NS = 2 * C::KS, NH = NS + 2 * C::MB;
  const int kb = f / NH, g = f % NH;
  const char *base = (const char *)smem;
  if (g < NS) {
    const unsigned o = so + 2u * 32u * D * (unsigned)kb;     // second half: rows 32..
    return *(const bf16x8 *)(base + ((g & 1) ? ad.vr[g >> 1] : ad.kr[g >> 1]) + o);
  }
  const int gq = g - NS;
  const unsigned o = so + 2u * D * (unsigned)(32 * kb + 16 * (gq / C::MB));
  return cat4(lds_read_tr4((const bf16 *)(base + ad.kt[gq % C::MB][0] + o)),
              lds_read_tr4((const bf16 *)(base + ad.kt[gq % C::MB][1] + o)));
}

// One 64-key tile, in two 32-key halves:
// S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - Delta), dQ^T += K^T dS^T
// (K^T read from the row-major K tile with transpose reads).  The products
// run in a fixed order, one per scheduling chunk, each chunk issuing the LDS
// operand PF products ahead; the softmax of a half sits between its S/dP and
// dQ products (the other wave on the SIMD keeps the matrix core busy then).
template <int D>
__device__ __forceinline__ void dq_tile(DqState<D> &st, const bf16 *smem, const DqAddr<D> &ad, unsigned so, int n0,
                                        int wq0, int qrow, int lane, float c) {
  using C = DqCfg<D>;
  constexpr int KS = C::KS, MB = C::MB;
  constexpr int NS = 2 * KS, NH = NS + 2 * MB, NP = 2 * NH;
  constexpr int PF = 3;
  const int h = lane >> 5;
  const bool diag = n0 + kFwdBN - 1 > wq0;   // tile straddles this wave's diagonal
  bf16x8 op[NP];
  f32x16 s, p;
  bf16x8 db[2];
#pragma unroll
  for (int f = 0; f < PF; ++f) op[f] = dq_operand<D>(f, smem, ad, so);
#pragma clang loop unroll(full)
  for (int pj = 0; pj < NP; ++pj) {
    if (pj + PF < NP) op[pj + PF] = dq_operand<D>(pj + PF, smem, ad, so);
    const int kb = pj / NH, g = pj % NH;
    if (g < NS) {
      if (g & 1) p = mfma32x32x16(op[pj], st.gf[g >> 1], g == 1 ? st.ndlt : p);
      else s = mfma32x32x16(op[pj], st.qf[g >> 1], g == 0 ? f32x16{} : s);
    } else {
      const int gq = g - NS;
      st.acc[gq % MB] = mfma32x32x16(op[pj], db[gq / MB], st.acc[gq % MB]);
    }
    if (g == NS - 1) {                          // softmax of this half
      if (diag) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const int key = n0 + 32 * kb + 8 * (i >> 2) + 4 * h + (i & 3);
          if (key > qrow) s[i] = -INFINITY;
        }
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float e = fast_exp2(s[i] * c - st.lse2);
        db[i >> 3][i & 7] = (bf16)(e * p[i]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// One dQ unit (launch slot `slot` of the unit list).  smem: K and V tiles,
// a four-stage ring: K of stage s at smem + s*TILE, V at smem + (4+s)*TILE,
// filled by untracked loads (as in the forward).
template <int D, bool G_F32>
__device__ __forceinline__ void dq_unit(const AttnArgs &a, int slot, bf16 *smem) {
  using C = DqCfg<D>;
  const int4 u = a.units[slot];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int m0 = u.y * C::BM;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const int64_t qhead = it.q_off + (int64_t)u.z * D;
  const bool loader = wave < C::NL;
  const TileLoader<D, C::BN, C::NL> ldK((const bf16 *)a.k + it.kv_off + (int64_t)u.w * D, ks, wave % C::NL, lane);
  const TileLoader<D, C::BN, C::NL> ldV((const bf16 *)a.v + it.kv_off + (int64_t)u.w * D, ks, wave % C::NL, lane);

  const int wq0 = m0 + wave * 32;
  const int qrow = wq0 + l32;
  const int n_end = min(L, m0 + C::BM);
  const int n_tiles = (n_end + C::BN - 1) / C::BN;
  const int wave_tiles = wq0 < L ? min(n_tiles, (wq0 + 31) / C::BN + 1) : 0;

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
    const float nd = a.delta[srow];          // -Delta
#pragma unroll
    for (int e = 0; e < 16; ++e) st.ndlt[e] = nd;
  }
  // The query-side registers land before the tile loads are issued: the
  // compiler does not count those loads, so a wait of its own for these
  // registers inside the loop would drain the ring.
  wait_all_loads();
  // tiles 0..2 in flight (past the item end a tile load fetches nothing)
  if (loader)
    for (int j = 0; j < 3; ++j) {
      ldK.load_untracked(smem + j * C::TILE, j * C::BN, L);
      ldV.load_untracked(smem + (4 + j) * C::TILE, j * C::BN, L);
    }
#pragma unroll
  for (int mb = 0; mb < C::MB; ++mb) st.acc[mb] = f32x16{};
  const float c = a.scale_log2;
  const DqAddr<D> ad(lane, 2u * 4u * C::TILE);
  constexpr unsigned TB = 2u * C::TILE;       // bytes per tile

  // step t: as in the forward -- wait for this wave's loads of tile t,
  // barrier, refill tile t-1's stage with tile t+3, process tile t
  int t = 0;
  for (;;) {
#define NSP_DQ_STEP(CUR, FILL)                                                      \
    {                                                                               \
      wait_loads_le<2 * C::LPW>();                                                  \
      stage_barrier();                                                              \
      if (loader) {                                                                 \
        ldK.load_untracked(smem + (FILL) * C::TILE, (t + 3) * C::BN, L);            \
        ldV.load_untracked(smem + (4 + (FILL)) * C::TILE, (t + 3) * C::BN, L);      \
      }                                                                             \
      if (t < wave_tiles)                                                           \
        dq_tile<D>(st, smem, ad, (CUR) * TB, t * C::BN, wq0, qrow, lane, c);        \
      if (++t >= n_tiles) break;                                                    \
    }
    NSP_DQ_STEP(0, 3)
    NSP_DQ_STEP(1, 0)
    NSP_DQ_STEP(2, 1)
    NSP_DQ_STEP(3, 2)
#undef NSP_DQ_STEP
  }
  // no buffer->LDS load may still be in flight when the workgroup ends
  wait_all_loads();

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

// dQ pass.  With queue heads (more units than compute units), one
// persistent workgroup per compute unit takes units from the per-XCD queues,
// as the dK/dV pass does; without (heads == nullptr), workgroup b runs launch
// slot b.
template <int D, bool G_F32>
__global__ void __launch_bounds__(64 * kFwdWaves, 1) bwd_dq_kernel(AttnArgs a, int *heads, int n_units) {
  __shared__ __attribute__((aligned(16))) bf16 smem[8 * DqCfg<D>::TILE];
  __shared__ int s_slot;
  const int own = (int)(__builtin_amdgcn_s_getreg(kHwRegXccId) % kXcdQueues);
  for (int iter = 0;; ++iter) {
    const int slot = heads ? next_queue_slot(heads, n_units, own, &s_slot) : (iter == 0 ? (int)blockIdx.x : -1);
    if (slot < 0) break;
    dq_unit<D, G_F32>(a, slot, smem);
  }
}

// ----------------------------------------------------------------- dK/dV --

template <int D>
struct KvCfg {
  static constexpr int BN = kBwdBN;          // keys per unit (4 waves x 32)
  static constexpr int BM = kBwdBM;          // query rows per step (one LDS stage)
  static constexpr int SUB = 32;             // query rows per sub-step
  static constexpr int QT = BM * D;          // elements of one Q or dO tile
  static constexpr int KS = D / 16;
  static constexpr int MB = D / 32;
  // one pipeline stage, in bf16 units: Q tile | dO tile | lse2[BM] | Delta[BM] (float)
  static constexpr int STAGE = 2 * QT + 4 * BM;
  // direct buffer->LDS loads per wave and stage (two tiles, lse2, Delta)
  static constexpr int LOADS = 2 * TileLoader<D, BM>::PER_WAVE + 2;
};

// The matrix products of the dK/dV steps, written out so that each value sits
// in the register file that uses it: S and dP accumulate in VGPRs (the vector
// units read them), dK^T and dV^T in AGPRs (read once, at the end), and K and
// V, the B operands of S and dP, stay in AGPRs.  Left to itself the compiler
// puts every product in AGPRs once the kernel needs more than 256 registers,
// and then copies S and dP to VGPRs, 64 copies per step.
// The compiler inserts no wait states for these products.  The schedule of
// kv_step keeps each S / dP result more than sixteen products from its first
// vector read, starts each S chain from the constant 0, waits two cycles
// before a dP chain reads its starting value, and the kernel waits before the
// epilogue reads dK / dV (kv_drain).  Accumulator chains (same registers in
// and out) need no wait.
__device__ __forceinline__ void kv_mma_s0(f32x16 &c, bf16x8 a, const bf16x8 &b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(c) : "v"(a), "a"(b));
}
__device__ __forceinline__ void kv_mma_p0(f32x16 &c, bf16x8 a, const bf16x8 &b) {
  asm volatile("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "a"(b));
}
__device__ __forceinline__ void kv_mma_v(f32x16 &c, bf16x8 a, const bf16x8 &b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c) : "v"(a), "a"(b));
}
__device__ __forceinline__ void kv_mma_acc(f32x16 &c, bf16x8 a, bf16x8 b) {
  asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(c) : "v"(a), "v"(b));
}

constexpr int kKvPf = 4;   // LDS operand prefetch distance of the dK/dV steps, in products

template <int D>
struct KvState {
  bf16x8 kf[D / 16];   // K (B operand of S = Q K^T: column = key, k = head_dim)
  bf16x8 vf[D / 16];   // V (B operand of dP = dO V^T)
  f32x16 dk[D / 32];   // dK^T (row = head_dim, column = key)
  f32x16 dv[D / 32];   // dV^T
  f32x16 s, p;         // S and dP of the sub-tile being finished (C layout)
  // read ahead by the previous sub-step, for the sub-tile whose S and dP the
  // next products compute: its -Delta (start of its dP products) and the LDS
  // operands of the first KV_PF products
  f32x16 pn0;
  bf16x8 op0[kKvPf];
};

// Cursor over the unit's (query tile, query head) steps: the heads of the
// group for one tile, then the next tile, tiles ascending from the diagonal
// or descending from the item end to it.  Pointers to the step's tile, moved
// on by additions.
template <int D>
struct KvCursor {
  TileLoader<D, kBwdBM> q, g;   // lane offsets and LDS slots of the tile loads
  const bf16 *pq, *pg;          // Q / dO: row m of the current query head
  const float *pl, *pd;         // lse2 / -Delta: entry m of the current query head
  int m;                        // first row of the tile
  int hh, nh;                   // current head (from the unit's first), heads of the unit
  int dm;                       // +BM or -BM: the next tile
  int64_t tq;                   // Q / dO elements from the last head of a tile to the first of the next
  int tl;                       // lse2 / -Delta entries, likewise
};

// The loads of one tile into one stage: Q and dO rows (PER_WAVE 16-byte
// loads each per wave), lse2 and -Delta (one 4-byte load each per wave; lane
// e fetches the entries of tile row e, zero past the item end, and the four
// waves write the same values).  They are untracked loads (the compiler adds
// no waits for them; the step's wait and barrier order them), one per chunk
// of the step's first chunks: issued together right after the barrier, the
// four waves' 40 loads would queue at the memory pipeline and stall every
// wave until its last one is taken; spread over the whole step they arrive
// later and the step is slower again (measured).
template <int D>
struct KvFill {
  static constexpr int PW = TileLoader<D, kBwdBM>::PER_WAVE;
  __amdgpu_buffer_rsrc_t rq, rg, rl, rd;
  int nq, nl;                   // bytes in range: Q / dO, lse2 / -Delta
  bf16 *stage;
};

// The fill of the cursor's tile is set up in three parts (byte ranges, the
// Q / dO resources, the lse2 / -Delta resources), and the cursor then moves
// on; the dK/dV steps spread these over chunks with room to spare.  A fill
// that is not `live` (past the unit's last tile: the stage is never read)
// gets empty ranges, so its loads write zeros and fetch nothing; every wave
// still issues the same loads on every step, so that no load hides behind a
// branch.
template <int D>
__device__ __forceinline__ void kv_fill_ranges(KvFill<D> &f, const KvCursor<D> &cu, bf16 *stage, int L,
                                               int row_bytes, bool live) {
  const int rows = live ? min(L - cu.m, kRsrcRows) : 0;
  f.nq = max(0, rows * row_bytes - (row_bytes - 2 * D));
  f.nl = max(0, rows) * 4;
  f.stage = stage;
  asm volatile("" : "+s"(f.nq), "+s"(f.nl));
}
template <int D>
__device__ __forceinline__ void kv_fill_qg(KvFill<D> &f, const KvCursor<D> &cu) {
  f.rq = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16 *>(cu.pq), 0, f.nq, 0x00020000);
  f.rg = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16 *>(cu.pg), 0, f.nq, 0x00020000);
  asm volatile("" : "+s"(f.rq), "+s"(f.rg));
}
template <int D>
__device__ __forceinline__ void kv_fill_ld(KvFill<D> &f, const KvCursor<D> &cu) {
  f.rl = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(cu.pl), 0, f.nl, 0x00020000);
  f.rd = __builtin_amdgcn_make_buffer_rsrc(const_cast<float *>(cu.pd), 0, f.nl, 0x00020000);
  asm volatile("" : "+s"(f.rl), "+s"(f.rd));
}
// Move the cursor to the next step: the next query head of the tile, or the
// first head of the next tile.  Past the unit's last step it keeps moving
// (its pointers then leave the item); the fills it sets up there are not
// live and access nothing.
template <int D>
__device__ __forceinline__ void kv_advance(KvCursor<D> &cu, int L) {
  if (++cu.hh < cu.nh) {
    cu.pq += D;
    cu.pg += D;
    cu.pl += L;
    cu.pd += L;
  } else {
    cu.hh = 0;
    cu.m += cu.dm;
    cu.pq += cu.tq;
    cu.pg += cu.tq;
    cu.pl += cu.tl;
    cu.pd += cu.tl;
  }
}

// A direct buffer->LDS load like load_lds_untracked, with the LDS address
// given as a register plus a constant: M0 is formed by one scalar add at the
// load, so that the kernel keeps one base per stage in registers rather than
// one address per load.  The add sets SCC (its carry), which the compiler is
// told.
template <int BYTES, unsigned OFF>
__device__ __forceinline__ void kv_load_lds(__amdgpu_buffer_rsrc_t rs, unsigned voff, unsigned lds_base) {
  static_assert(BYTES == 4 || BYTES == 16, "load size");
  if constexpr (BYTES == 16)
    asm volatile("s_add_u32 m0, %0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(lds_base), "v"(voff), "s"(rs), "i"(OFF)
                 : "memory", "scc");
  else
    asm volatile("s_add_u32 m0, %0, %3\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(lds_base), "v"(voff), "s"(rs), "i"(OFF)
                 : "memory", "scc");
}

template <typename T>
__device__ __forceinline__ unsigned lds_addr(const T *p) {
  return (unsigned)(uintptr_t)(__attribute__((address_space(3))) const void *)p;
}

// Issue load J (0 .. LOADS-1) of a fill.
template <int D, int J>
__device__ __forceinline__ void kv_fill_issue(const KvFill<D> &f, const KvCursor<D> &cu) {
  using C = KvCfg<D>;
  using TL = TileLoader<D, kBwdBM>;
  constexpr int PW = KvFill<D>::PW;
  const unsigned vl = (unsigned)(threadIdx.x & 63) * 4;
  // this wave's slots of the stage; the lse2 / -Delta rows, which every wave
  // writes alike
  const unsigned wbase = lds_addr(cu.q.dst(f.stage, 0)), sbase = lds_addr(f.stage);
  if constexpr (J < PW) kv_load_lds<16, 2u * J * TL::RPI * D>(f.rq, cu.q.voff[J], wbase);
  else if constexpr (J < 2 * PW) kv_load_lds<16, 2u * (C::QT + (J - PW) * TL::RPI * D)>(f.rg, cu.g.voff[J - PW], wbase);
  else if constexpr (J == 2 * PW) kv_load_lds<4, 2u * 2 * C::QT>(f.rl, vl, sbase);
  else kv_load_lds<4, 2u * (2 * C::QT + 2 * C::BM)>(f.rd, vl, sbase);
}

// Load j of a fill, j known once the caller's loop is unrolled.
template <int D, int J = 0>
__device__ __forceinline__ void kv_fill_issue_rt(const KvFill<D> &f, const KvCursor<D> &cu, int j) {
  if constexpr (J < KvCfg<D>::LOADS) {
    if (j == J) kv_fill_issue<D, J>(f, cu);
    else kv_fill_issue_rt<D, J + 1>(f, cu, j);
  }
}

// Set up the fill of the cursor's tile into `stage`, move the cursor on.
template <int D>
__device__ __forceinline__ KvFill<D> kv_fill(KvCursor<D> &cu, bf16 *stage, int L, int row_bytes, bool live) {
  KvFill<D> f;
  kv_fill_ranges<D>(f, cu, stage, L, row_bytes, live);
  kv_fill_qg<D>(f, cu);
  kv_fill_ld<D>(f, cu);
  kv_advance<D>(cu, L);
  return f;
}

// Issue all loads of the cursor's tile into a stage, move the cursor on.
template <int D>
__device__ __forceinline__ void kv_issue(KvCursor<D> &cu, bf16 *stage, int L, int row_bytes, bool live) {
  const KvFill<D> f = kv_fill<D>(cu, stage, L, row_bytes, live);
#pragma unroll
  for (int j = 0; j < KvCfg<D>::LOADS; ++j) kv_fill_issue_rt<D>(f, cu, j);
}

// What a step's second sub-step sets up for the next step: the fill of
// `stage` (live or not) from the cursor, which it then moves on.
template <int D>
struct KvNext {
  KvCursor<D> &cu;
  bf16 *stage;
  int L, row_bytes;
  bool live;
};

// -Delta of the rows that the 16 accumulator elements of this lane hold
// (rows 8g + 4h .. 8g + 4h + 3 of element block g), from the lse2 / -Delta
// block `ld` of a sub-tile: the starting value of its dP products, which
// then end at dP - Delta.
template <int D>
__device__ __forceinline__ f32x16 kv_ndelta(const float *ld, int lane) {
  const float *r = ld + KvCfg<D>::BM + 4 * (lane >> 5);
  const f32x4 a0 = *(const f32x4 *)(r), a1 = *(const f32x4 *)(r + 8), a2 = *(const f32x4 *)(r + 16),
              a3 = *(const f32x4 *)(r + 24);
  return f32x16{a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3],
                a2[0], a2[1], a2[2], a2[3], a3[0], a3[1], a3[2], a3[3]};
}

// S and dP of the query tile held (row-major) in `stage`.
template <int D>
__device__ __forceinline__ void kv_scores(const KvState<D> &st, const bf16 *stage, int lane, f32x16 &s,
                                          f32x16 &p) {
  using C = KvCfg<D>;
  const int l32 = lane & 31, h = lane >> 5;
  s = f32x16{};
  p = kv_ndelta<D>((const float *)(stage + 2 * C::QT), lane);
#pragma unroll
  for (int k = 0; k < C::KS; ++k) {
    const int o = tile_off<D>(l32, 16 * k + 8 * h);
    s = mfma32x32x16(*(const bf16x8 *)(stage + o), st.kf[k], s);
    p = mfma32x32x16(*(const bf16x8 *)(stage + C::QT + o), st.vf[k], p);
  }
}

// LDS operand of product f of a sub-step: f < 2*KS: row operand of the next
// sub-tile for S = Q K^T (even f) or dP = dO V^T (odd f), k block f/2; then
// the 2*MB dV^T products (transposed dO of this sub-tile), then the 2*MB dK^T
// products (transposed Q), each with k block kk = g/MB and head_dim block
// md = g%MB for g counted within its group.
template <int D>
__device__ __forceinline__ bf16x8 kv_operand(int f, const bf16 *cur, const bf16 *nxt, int lane) {
  using C = KvCfg<D>;
  constexpr int NS = 2 * C::KS, NDV = 2 * C::MB;
  if (f < NS) {
    const int o = tile_off<D>(lane & 31, 16 * (f >> 1) + 8 * (lane >> 5));
    return *(const bf16x8 *)(nxt + ((f & 1) ? C::QT : 0) + o);
  }
  const int g = f - NS;
  const bool dv = g < NDV;
  const int gg = dv ? g : g - NDV;
  return lds_tr_operand<D>(dv ? cur + C::QT : cur, 16 * (gg / C::MB), 32 * (gg % C::MB), lane);
}

// One sub-step of the software pipeline, over 32 query rows.  On entry
// st.s / st.p hold S and dP of sub-tile j (whose Q and dO rows start at `cur`
// in a stage, its lse2 / -Delta at cur_ld); `nxt` is sub-tile j+1 (the other
// half of the stage or the first half of the next one), `nn` / nn_ld sub-tile
// j+2; st.pn0 and st.op0 hold the -Delta of sub-tile j+1 and the operands of
// the first products.  The sub-step
//   * sets S to -inf where the query row precedes the key or lies past the
//     item end (only on the diagonal and tail sub-tiles),
//   * computes S and dP of sub-tile j+1 on the matrix cores while the vector
//     units turn sub-tile j into P = exp2(c S - lse2) and dS = P (dP - Delta),
//   * accumulates dV^T += dO^T P and dK^T += Q^T dS (dO^T, Q^T by transpose
//     reads at `cur`), leaves S and dP of sub-tile j+1 in st.s / st.p, and
//     the -Delta and first operands of sub-tile j+2 in st.pn0 / st.op0.
// The 2*KS + 4*MB products (S/dP of sub-tile j+1, then dV^T, then dK^T of
// sub-tile j) run as a fixed sequence of chunks: chunk j issues the LDS
// operand of product j+PF (for the last chunks, one of the next sub-step) and
// runs product j, so that no product waits for an operand read issued just
// before it, also across sub-steps.  The vector work goes by pairs of
// elements in small independent pieces placed beside the products, at most
// about five instructions per product (what one wave issues while its matrix
// product runs): scale and shift, exp2, and packing P to bf16 beside the S/dP
// products; the product with P (dP - Delta comes out of the matrix core, its
// chain having started from -Delta) and packing dS beside the dV products
// (dS is first needed by the dK products); the reads of the next -Delta
// beside the dK products.  A scheduling fence after each chunk keeps that
// order.
// After the last sub-tile the scores of the following stage are computed and
// dropped (a read of stale LDS contents, never used).
template <int D, int SUB>
__device__ __forceinline__ void kv_step(KvState<D> &st, const bf16 *cur, const float *cur_ld, const bf16 *nxt,
                                        const bf16 *nn, const float *nn_ld, int m0, int key, int L, int lane,
                                        float c, KvFill<D> &fill, const KvNext<D> &nx) {
  using C = KvCfg<D>;
  constexpr int NS = 2 * C::KS;     // S / dP products of sub-tile j+1
  constexpr int NDV = 2 * C::MB;    // dV^T products (then as many dK^T products)
  constexpr int NP = NS + 2 * NDV;
  constexpr int PF = kKvPf;
  constexpr int ND = NS + NDV;      // chunks ND .. ND+3 read the next -Delta
  static_assert(PF < NS && ND + 4 <= NP, "prefetch schedule");
  const int l32 = lane & 31, h = lane >> 5;
  if (m0 < key - l32 + 31 || m0 + C::SUB > L) {
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int q = m0 + 8 * (i >> 2) + 4 * h + (i & 3);
      if (q < key || q >= L) st.s[i] = -INFINITY;
    }
  }
  bf16x8 op[NP + PF];
#pragma unroll
  for (int f = 0; f < PF; ++f) op[f] = st.op0[f];
  // the dP products of sub-tile j+1 start from its -Delta (and end at
  // dP - Delta)
  f32x16 sn, pn = st.pn0, pnn;
  f32x4 nd4[4];
  const float *ndrow = nn_ld + C::BM + 4 * h;
  bf16x8 pb[2], db[2];
  float t[16], x[16];
  // chunk of the scale-and-shift of element pair q (exp2 one chunk later,
  // the bf16 pack of P two chunks later), and of the dS of pair q.  These
  // products get no wait states from the compiler: a vector result needs two
  // wait states before a matrix product reads it, so every pack lands at
  // least two chunks before the first product that reads its half of P or dS.
  constexpr int SPAN = NS < 8 * (NS + C::MB - 4) / 7 ? NS : 8 * (NS + C::MB - 4) / 7;
  constexpr auto pa = [](int q) { return q * SPAN / 8; };
  constexpr auto pd = [](int q) { return NS + q * NDV / 8; };
  static_assert(pa(3) + 4 <= NS && pa(7) + 4 <= NS + C::MB, "P packed two chunks before its dV products");
  static_assert(pd(3) + 2 <= NS + NDV && pd(7) + 2 <= NS + NDV + C::MB, "dS packed two chunks before its dK products");
  // lse2 of the rows that element block g holds in this lane (rows
  // 8g + 4h .. 8g + 4h + 3), read from the stage two chunks before first use
  // (before the chunks when that is earlier than the first)
  f32x4 l4[4];
  const float *lrow = cur_ld + 4 * h;
#pragma unroll
  for (int g = 0; g < 4; ++g)
    if (pa(2 * g) < 2) l4[g] = *(const f32x4 *)(lrow + 8 * g);
#pragma clang loop unroll(full)
  for (int pj = 0; pj < NP; ++pj) {            // chunk pj runs product pj
    if (pj + PF < NP) op[pj + PF] = kv_operand<D>(pj + PF, cur, nxt, lane);
    else op[pj + PF] = kv_operand<D>(pj + PF - NP, cur, nn, lane);
    // one LDS wait per two products: at even chunks the wait also covers the
    // operand of the next chunk (read one chunk after this one's), so the
    // odd chunk's product issues without one (0.9% faster than a wait per
    // product; a wait per four products stalls: 8% slower)
    if (!(pj & 1) && pj + 1 < NP) asm volatile("" :: "v"(op[pj + 1]));
    if (pj < NS) {
      if (pj == 0) kv_mma_s0(sn, op[pj], st.kf[0]);
      else if (pj == 1) kv_mma_p0(pn, op[pj], st.vf[0]);
      else if (pj & 1) kv_mma_v(pn, op[pj], st.vf[pj >> 1]);
      else kv_mma_v(sn, op[pj], st.kf[pj >> 1]);
    } else if (pj < NS + NDV) {
      const int g = pj - NS;
      kv_mma_acc(st.dv[g % C::MB], op[pj], pb[g / C::MB]);
    } else {
      const int g = pj - NS - NDV;
      kv_mma_acc(st.dk[g % C::MB], op[pj], db[g / C::MB]);
    }
#pragma unroll
    for (int g = 0; g < 4; ++g)
      if (pa(2 * g) >= 2 && pj == pa(2 * g) - 2) l4[g] = *(const f32x4 *)(lrow + 8 * g);
    if (pj >= ND && pj < ND + 4) nd4[pj - ND] = *(const f32x4 *)(ndrow + 8 * (pj - ND));
#pragma unroll
    for (int q = 0; q < 8; ++q) {               // element pair (2q, 2q+1)
      const int sa = pa(q);                     // P: chunks sa .. sa+2
      const int sb = pd(q);                     // dS: chunk sb
#pragma unroll
      for (int e = 2 * q; e < 2 * q + 2; ++e) {
        if (pj == sa) t[e] = st.s[e] * c - l4[e >> 2][e & 3];
        if (pj == sa + 1) x[e] = fast_exp2(t[e]);
        if (pj == sa + 2) pb[e >> 3][e & 7] = (bf16)x[e];
        if (pj == sb) db[e >> 3][e & 7] = (bf16)(x[e] * st.p[e]);
      }
    }
    // the step's tile loads, one per chunk in the first chunks of the step
    // (issued together right after the barrier, the four waves' loads queue
    // at the memory pipeline, which takes one about every 12 cycles, and
    // every wave stalls until its last one is taken)
    if constexpr (SUB == 0)
      if (pj < C::LOADS) kv_fill_issue_rt<D>(fill, nx.cu, pj);
    // the fill of the next step, in parts beside the dK products
    if constexpr (SUB == 1) {
      constexpr int F0 = NS + NDV, FS = NDV / 4;
      if (pj == F0) kv_fill_ranges<D>(fill, nx.cu, nx.stage, nx.L, nx.row_bytes, nx.live);
      if (pj == F0 + FS) kv_fill_qg<D>(fill, nx.cu);
      if (pj == F0 + 2 * FS) kv_fill_ld<D>(fill, nx.cu);
      if (pj == F0 + 3 * FS) kv_advance<D>(nx.cu, nx.L);
    }
    __builtin_amdgcn_sched_barrier(0);
  }
#pragma unroll
  for (int g = 0; g < 4; ++g)
#pragma unroll
    for (int i = 0; i < 4; ++i) pnn[4 * g + i] = nd4[g][i];
  st.s = sn;
  st.p = pn;
  st.pn0 = pnn;
#pragma unroll
  for (int f = 0; f < PF; ++f) st.op0[f] = op[NP + f];
}

// Wait until the last dK^T / dV^T products have written their registers
// before anything reads them (the compiler does not see those products).
template <int D>
__device__ __forceinline__ void kv_drain(KvState<D> &st) {
  static_assert(D / 32 == 4 || D / 32 == 2, "head_dim");
  if constexpr (D / 32 == 4)
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(st.dk[0]), "+a"(st.dk[1]), "+a"(st.dk[2]), "+a"(st.dk[3]), "+a"(st.dv[0]), "+a"(st.dv[1]),
                   "+a"(st.dv[2]), "+a"(st.dv[3]));
  else
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7"
                 : "+a"(st.dk[0]), "+a"(st.dk[1]), "+a"(st.dv[0]), "+a"(st.dv[1]));
}

// One dK/dV unit (launch slot `slot` of the unit list) on the workgroup's
// four LDS pipeline stages.
template <int D, bool G_F32>
__device__ __forceinline__ void dkdv_unit(const AttnArgs &a, int slot, bf16 *stg0, bf16 *stg1, bf16 *stg2,
                                          bf16 *stg3) {
  using C = KvCfg<D>;
  const int4 u = a.units[slot];
  const ItemDesc it = a.items[u.x];
  const int L = it.L;
  const int n0 = (u.y & kKvTileMask) * C::BN;
  const bool desc = (u.y & kKvDescending) != 0;
  const int i_lo = u.z & 0xffff, i_hi = u.z >> 16;
  const int wave = wave_id(), lane = threadIdx.x & 63;
  const int l32 = lane & 31, h = lane >> 5;
  const int64_t qs = (int64_t)it.hq * D;
  const int64_t ks = (int64_t)it.hkv * D;
  const int64_t kvhead = it.kv_off + (int64_t)u.w * D;

  const int kbase = n0 + wave * 32;           // first key of this wave
  const int key = kbase + l32;                // this lane's key (MFMA column)
  const int mt0 = n0 / C::BM;                     // first query tile touching the keys
  const int mt_end = (L + C::BM - 1) / C::BM;
  const int nh = i_hi - i_lo;
  const int n_iter = nh * (mt_end - mt0);

  KvState<D> st;
  {
    const int64_t r = kvhead + (int64_t)min(key, L - 1) * ks + 8 * h;
#pragma unroll
    for (int k = 0; k < C::KS; ++k) {
      st.kf[k] = *(const bf16x8 *)((const bf16 *)a.k + r + 16 * k);
      st.vf[k] = *(const bf16x8 *)((const bf16 *)a.v + r + 16 * k);
    }
    // K and V move to AGPRs here, once (they are the B operands of every S and
    // dP product, which reads them from there)
#pragma unroll
    for (int k = 0; k < C::KS; ++k) {
      asm volatile("" : "+a"(st.kf[k]));
      asm volatile("" : "+a"(st.vf[k]));
    }
  }
#pragma unroll
  for (int md = 0; md < C::MB; ++md) { st.dk[md] = f32x16{}; st.dv[md] = f32x16{}; }
  const float c = a.scale_log2;

  // A group without query heads (n_iter = 0) still runs the prologue: its
  // fills are empty (zeros, nothing fetched) and the steps that follow are
  // skipped, so the unit writes zero gradients.
  const int m_first = (desc ? mt_end - 1 : mt0) * C::BM;
  const int dm = desc ? -C::BM : C::BM;
  const int row_bytes = (int)qs * 2;
  KvCursor<D> cu{TileLoader<D, C::BM>((const bf16 *)a.q, qs, wave, lane),
                 TileLoader<D, C::BM>((const bf16 *)a.dout, qs, wave, lane)};
  cu.pq = (const bf16 *)a.q + it.q_off + (int64_t)m_first * qs + (int64_t)i_lo * D;
  cu.pg = (const bf16 *)a.dout + it.q_off + (int64_t)m_first * qs + (int64_t)i_lo * D;
  cu.pl = a.lse2 + it.lse_off + (int64_t)i_lo * L + m_first;
  cu.pd = a.delta + it.lse_off + (int64_t)i_lo * L + m_first;
  cu.m = m_first;
  cu.hh = 0;
  cu.nh = nh;
  cu.dm = dm;
  cu.tq = (int64_t)dm * qs - (int64_t)(nh - 1) * D;
  cu.tl = dm - (nh - 1) * L;
  // prologue: steps 0..2 in flight
  kv_issue<D>(cu, stg0, L, row_bytes, 0 < n_iter);
  kv_issue<D>(cu, stg1, L, row_bytes, 1 < n_iter);
  kv_issue<D>(cu, stg2, L, row_bytes, 2 < n_iter);
  // the fill of the first step (step 3)
  KvFill<D> fill = kv_fill<D>(cu, stg3, L, row_bytes, 3 < n_iter);
  __builtin_amdgcn_s_waitcnt(0);               // tiles 0..2, K and V landed
  stage_barrier();
  {
    // moved into VGPRs (compiler-made copies, which wait for the matrix
    // core), like the S and dP the steps hand over: the loop-carried values
    // then stay in VGPRs instead of being copied back and forth each step
    f32x16 s0, p0;
    kv_scores<D>(st, stg0, lane, s0, p0);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      st.s[e] = pin(s0[e]);
      st.p[e] = pin(p0[e]);
    }
    st.pn0 = kv_ndelta<D>((const float *)(stg0 + 2 * C::QT) + C::SUB, lane);
#pragma unroll
    for (int f = 0; f < kKvPf; ++f) st.op0[f] = kv_operand<D>(f, stg0, stg0 + C::SUB * D, lane);
  }
  int m0 = m_first, mh = 0;
  for (int i = 0; i < n_iter;) {
#define NSP_KV_STEP(CUR, NXT)                                                                     \
    {                                                                                             \
      wait_loads_le<C::LOADS>();                                                                  \
      stage_barrier();                                                                            \
      const KvNext<D> nx{cu, CUR, L, row_bytes, i + 4 < n_iter};                                \
      kv_step<D, 0>(st, CUR, (const float *)(CUR + 2 * C::QT), CUR + C::SUB * D, NXT,               \
                    (const float *)(NXT + 2 * C::QT), m0, key, L, lane, c, fill, nx);                 \
      kv_step<D, 1>(st, CUR + C::SUB * D, (const float *)(CUR + 2 * C::QT) + C::SUB, NXT,             \
                    NXT + C::SUB * D, (const float *)(NXT + 2 * C::QT) + C::SUB, m0 + C::SUB, key, L,  \
                    lane, c, fill, nx);                                                             \
      if (++mh == nh) {                                                                           \
        mh = 0;                                                                                   \
        m0 += dm;                                                                                 \
      }                                                                                           \
      if (++i == n_iter) break;                                                                   \
    }
    // step i (64 query rows, two sub-steps): wait for tile i+1; the loads of
    // tile i+3 go to the stage of tile i-1, and the second sub-step sets up
    // the fill of the next step (tile i+4, into the stage of tile i)
    NSP_KV_STEP(stg0, stg1)
    NSP_KV_STEP(stg1, stg2)
    NSP_KV_STEP(stg2, stg3)
    NSP_KV_STEP(stg3, stg0)
#undef NSP_KV_STEP
  }

  kv_drain<D>(st);
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

// dK/dV pass.  With queue heads (more units than compute units), one
// persistent workgroup per compute unit takes units from the per-XCD queues,
// stored one after another (a.qoff; next_range_slot); without
// (heads == nullptr), workgroup b runs launch slot b.
template <int D, bool G_F32>
__global__ void __launch_bounds__(256, 1) bwd_dkdv_kernel(AttnArgs a, int *heads, int n_units) {
  using C = KvCfg<D>;
  // four pipeline stages (distinct objects, so that the compiler can tell the
  // stage being filled from the ones being read)
  __shared__ __attribute__((aligned(16))) bf16 stg0[C::STAGE];
  __shared__ __attribute__((aligned(16))) bf16 stg1[C::STAGE];
  __shared__ __attribute__((aligned(16))) bf16 stg2[C::STAGE];
  __shared__ __attribute__((aligned(16))) bf16 stg3[C::STAGE];
  __shared__ int s_slot;
  const int own = (int)(__builtin_amdgcn_s_getreg(kHwRegXccId) % kXcdQueues);
  for (int iter = 0;; ++iter) {
    const int slot = heads ? next_range_slot(heads, a.qoff, own, &s_slot) : (iter == 0 ? (int)blockIdx.x : -1);
    if (slot < 0) break;
    dkdv_unit<D, G_F32>(a, slot, stg0, stg1, stg2, stg3);
    // nothing may still be loading into the stages when the next unit fills them
    __builtin_amdgcn_s_waitcnt(0);
  }
}

}  // namespace

hipError_t launch_bwd_preprocess(int head_dim, bool o_f32, const AttnArgs &a, int n_blocks, hipStream_t s) {
  if (n_blocks == 0) return hipSuccess;
  dim3 grid(n_blocks), block(256);
  if (head_dim == 128) {
    if (o_f32) bwd_preprocess_kernel<128, true><<<grid, block, 0, s>>>(a);
    else bwd_preprocess_kernel<128, false><<<grid, block, 0, s>>>(a);
  } else {
    if (o_f32) bwd_preprocess_kernel<64, true><<<grid, block, 0, s>>>(a);
    else bwd_preprocess_kernel<64, false><<<grid, block, 0, s>>>(a);
  }
  return hipGetLastError();
}

// Grid and queue heads of a pass over n_units units: with more units than
// compute units, one persistent workgroup per compute unit (the kernels'
// resources allow no more) and the heads; otherwise one workgroup per unit
// and no heads.
static hipError_t pass_grid(int n_units, int *heads_if_persistent, dim3 *grid, int **heads) {
  int cus = 0;
  hipError_t e = compute_units(&cus);
  if (e != hipSuccess) return e;
  const bool persistent = n_units > cus;
  *grid = dim3(persistent ? cus : n_units);
  *heads = persistent ? heads_if_persistent : nullptr;
  return hipSuccess;
}

hipError_t launch_bwd_dq(int head_dim, bool g_f32, const AttnArgs &a, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  dim3 grid, block(64 * kFwdWaves);
  int *heads = nullptr;
  hipError_t e = pass_grid(n_units, a.queue + kDqQueue0, &grid, &heads);
  if (e != hipSuccess) return e;
  if (head_dim == 128) {
    if (g_f32) bwd_dq_kernel<128, true><<<grid, block, 0, s>>>(a, heads, n_units);
    else bwd_dq_kernel<128, false><<<grid, block, 0, s>>>(a, heads, n_units);
  } else {
    if (g_f32) bwd_dq_kernel<64, true><<<grid, block, 0, s>>>(a, heads, n_units);
    else bwd_dq_kernel<64, false><<<grid, block, 0, s>>>(a, heads, n_units);
  }
  return hipGetLastError();
}

hipError_t launch_bwd_dkdv(int head_dim, bool g_f32, const AttnArgs &a, int n_units, hipStream_t s) {
  if (n_units == 0) return hipSuccess;
  dim3 grid, block(256);
  int *heads = nullptr;
  hipError_t e = pass_grid(n_units, a.queue + kKvQueue0, &grid, &heads);
  if (e != hipSuccess) return e;
  if (head_dim == 128) {
    if (g_f32) bwd_dkdv_kernel<128, true><<<grid, block, 0, s>>>(a, heads, n_units);
    else bwd_dkdv_kernel<128, false><<<grid, block, 0, s>>>(a, heads, n_units);
  } else {
    if (g_f32) bwd_dkdv_kernel<64, true><<<grid, block, 0, s>>>(a, heads, n_units);
    else bwd_dkdv_kernel<64, false><<<grid, block, 0, s>>>(a, heads, n_units);
  }
  return hipGetLastError();
}

}  // namespace nsp
