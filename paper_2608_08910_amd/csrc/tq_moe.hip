// Routed-expert MoE layer over folded tq experts: the dot pass of Sec. 2.2 applied to the
// gate, up and down projections of every routed expert (the paper's model has 43 such
// layers x 3 projections x 256 experts, Sec. 2.1). The glue around the projections
// (SiLU(gate) * up, the requantized hidden, the softmax-weighted sum after down) is the
// workload's definition, stated in tq.h.
//
// Stages (one kernel each, all on the caller's stream; no host synchronization):
//   prologue  quantize x per 256-block, and (one extra workgroup) dispatch the routing:
//             per-expert slot counts, the active-expert list (hottest first when a step
//             has several tokens), slot lists grouped by expert, task counts.
//   gate_up   static work queue over (active expert, row tile), tasks in rank order
//             strided over the grid (no atomics: a device-scope counter serializes
//             at one address across the 8 XCDs): a wave loads RPW rows of
//             gate and of up (each byte read once per step), walks the expert's tokens NT
//             at a time, and writes h = SiLU(g) * u per slot.
//   requant   quantize h per 256-block (same quantizer as x).
//   down      the same queue over (active expert, row tile) of the down projection,
//             writing y[slot][row].
//   combine   out[t] = sum_j w[t][j] * y[t*topk + j] in ascending j (fixed order: no
//             floating-point atomics, bitwise reproducible).
#include <hip/hip_ext.h>

#include <algorithm>
#include <atomic>
#include <mutex>
#include <type_traits>

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr int kMaxExperts = 4096;
constexpr int kMaxTopk = 64;
constexpr int kNumStages = 5;
static const char* const kStageNames[kNumStages] = {"prologue", "gate_up", "requant", "down", "combine"};

// Control words at the start of the workspace.
enum Ctrl {
  kFlags = 0, kNActive = 1, kTasksGU = 2, kTasksDn = 3, kNValid = 4, kTasksMGU = 5, kTasksMDn = 6,
  kTSmall = 7, kTasksMGUs = 8, kTasksMDns = 9, kTSingle = 10, kRSkip = 11, kCtrlWords = 64
};

constexpr int kMT = 128;     // tokens per MFMA task tile (eight 16-row MFMA tiles)
constexpr int kMWaves = 8;   // waves per MFMA workgroup, 16 weight rows each
constexpr int kMN = 16 * kMWaves;  // weight rows per MFMA task tile
constexpr int kMStages = 3;  // token-tile blocks in flight in LDS per MFMA workgroup
// Experts with at most kMTs slots (most of them at prefill under Zipf routing) run as a
// second MFMA launch with kMTs-token tiles and kMWavesS-wave workgroups: several such
// workgroups share a compute unit, so one's loads, MFMAs and epilogue overlap another's.
constexpr int kMTs = 32;
constexpr int kMWavesS = 4;
constexpr int kMNs = 16 * kMWavesS;
constexpr int64_t kMfmaMinSlots = 2048;  // automatic path choice: MFMA from this many slots
// Mixed path (automatic choice below kMfmaMinSlots slots, more than kHybMin tokens): the
// experts of more than kHybMin and at most kMTs slots run on the kMTs-token MFMA kernel
// beside the grouped VALU kernel, which takes the others. On the VALU kernel such an
// expert's task walks its tokens two at a time, every group's activation loads queued
// behind the compute unit's weight loads; on MFMA its tokens share one pass over the
// weights.
constexpr int kHybMin = 2;  // (measured on MI355X: 2 and 3 best at 8 and 32 tokens per step)
constexpr int kTbWaves = 4;  // waves per grouped VALU workgroup

struct Layout {
  size_t ctrl, active, act_off, tt_off, tile_exp, tt32_off, tile32_exp, slot_list, xq, xd, xb, h, hq, hd, hb, yd, total;
  // debug stage dump (TQ_MOE_DEBUG_STAGES), past `total`: g and u per slot, and the exact
  // block sums of gate, up (per slot, row, hidden block) and down (per slot, row, inter block)
  size_t dg, du, dgs, dus, dds, total_dbg;
};

static size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

static Layout make_layout(int n_experts, int hidden, int inter, int64_t t, int topk) {
  Layout L{};
  const size_t S = (size_t)t * topk;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  L.ctrl = take(kCtrlWords * 4);
  L.active = take((size_t)n_experts * 4);
  L.act_off = take(((size_t)n_experts + 1) * 4);
  L.tt_off = take(((size_t)n_experts + 1) * 4);
  L.tile_exp = take((S / kMT + (size_t)n_experts + 1) * 4);
  L.tt32_off = take(((size_t)n_experts + 1) * 4);
  L.tile32_exp = take((S / kMTs + (size_t)n_experts + 1) * 4);
  L.slot_list = take(S * 4);
  L.xq = take((size_t)t * hidden);
  L.xd = take((size_t)t * (hidden / 256) * 4);
  L.xb = take((size_t)t * (hidden / 256) * 4);
  L.h = take(S * inter * 4);
  L.hq = take(S * inter);
  L.hd = take(S * (inter / 256) * 4);
  L.hb = take(S * (inter / 256) * 4);
  L.yd = take(S * hidden * 4);
  L.total = o;
  L.dg = take(S * inter * 4);
  L.du = take(S * inter * 4);
  L.dgs = take(S * inter * (hidden / 256) * 4);
  L.dus = take(S * inter * (hidden / 256) * 4);
  L.dds = take(S * hidden * (inter / 256) * 4);
  L.total_dbg = o;
  return L;
}

// ---------------------------------------------------------------------------------
// Shared pieces
// ---------------------------------------------------------------------------------

// Quantize 8 consecutive 256-blocks per wave of the flattened block grid.
__device__ __forceinline__ void quantize_wave_blocks(const float* __restrict__ x, int64_t nblocks, int64_t wave_id,
                                                     int8_t* __restrict__ q, float* __restrict__ d,
                                                     int32_t* __restrict__ bsum) {
  const int lane = threadIdx.x & 63;
  const int64_t blk = wave_id * 8 + (lane >> 3);
  if (blk >= nblocks) return;
  const int cp = lane & 7;
  const float4* xp = reinterpret_cast<const float4*>(x + blk * 256 + cp * 32);
  float v[32];
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const float4 f = xp[m];
    v[4 * m + 0] = f.x;
    v[4 * m + 1] = f.y;
    v[4 * m + 2] = f.z;
    v[4 * m + 3] = f.w;
  }
  int qw[8], qs, bs;
  float dd;
  quantize_group32(v, qw, qs, dd, bs);
  int4* qp = reinterpret_cast<int4*>(q + blk * 256 + cp * 32);
  qp[0] = make_int4(qw[0], qw[1], qw[2], qw[3]);
  qp[1] = make_int4(qw[4], qw[5], qw[6], qw[7]);
  if (cp == 0) {
    d[blk] = dd;
    bsum[blk] = bs;
  }
}

// One matrix of one expert as buffer resources (codes and scales).
struct MatRsrc {
  __amdgpu_buffer_rsrc_t codes, scales;
};

__device__ __forceinline__ MatRsrc mat_rsrc(const uint8_t* codes, const uint16_t* scales, int n, int kb) {
  return {make_rsrc(codes, (uint32_t)n * (uint32_t)kb * 128u), make_rsrc(scales, (uint32_t)n * (uint32_t)kb * 2u)};
}

__device__ __forceinline__ float silu_f32(float z) { return z / (1.0f + expf(-z)); }

struct MoeArgs {
  int n_experts, hidden, inter, topk;
  int64_t t;
  const uint8_t* codes[3];
  const uint16_t* scales[3];
  int64_t stride_codes[3], stride_scales[3];
  const int32_t* topk_idx;
  const float* topk_w;
  int32_t* ctrl;
  int32_t* active;
  int32_t* act_off;
  int32_t* tt_off;  // per active expert: first token tile (kMT tokens) of the MFMA path
  int32_t* tile_exp;  // per token tile of the MFMA path: its active expert's rank
  int32_t* tt32_off;    // mixed path: per active expert, its first kMTs-token tile
  int32_t* tile32_exp;  // mixed path: per kMTs-token tile (experts of more than hyb slots), the rank
  int32_t* slot_list;
  int8_t* xq;
  float* xd;
  int32_t* xb;
  float* h;
  int8_t* hq;
  float* hd;
  int32_t* hb;
  float* yd;
  // debug stage dump: all null unless TQ_MOE_DEBUG_STAGES (a kernel-argument test, the same
  // for every lane and wave, so the kernels take one uniform branch around each store)
  float* dbg_g;
  float* dbg_u;
  int32_t* dbg_gsum;  // [slot][inter][hidden / 256]
  int32_t* dbg_usum;  // [slot][inter][hidden / 256]
  int32_t* dbg_dsum;  // [slot][hidden][inter / 256]
  int tiles_gu, tiles_dn;    // row tiles of the VALU kernels
  int tiles_mgu, tiles_mdn;  // row tiles of the MFMA kernels
  int tiles_mgus, tiles_mdns;  // row tiles of the small-tile MFMA kernels
  int hyb;  // mixed path: experts of more than hyb and at most kMTs slots go to MFMA (0: off)
};

// ---------------------------------------------------------------------------------
// prologue: dispatch (workgroup 0, dispatched first so that it runs beside the
// quantization rather than after it) + quantize x (workgroups 1 .. nq)
// ---------------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_moe_prologue(const float* __restrict__ x, MoeArgs A) {
  if (blockIdx.x > 0) {
    const int64_t nblocks = A.t * (A.hidden / 256);
    quantize_wave_blocks(x, nblocks, (int64_t)(blockIdx.x - 1) * 4 + (threadIdx.x >> 6), A.xq, A.xd, A.xb);
    return;
  }
  __shared__ int s_cnt[kMaxExperts];   // slots per expert
  __shared__ __attribute__((aligned(16))) int s_base[kMaxExperts];  // rank key, then the slot cursor
  __shared__ int s_ebr[kMaxExperts];   // expert of each rank
  __shared__ int s_scan[256], s_scan2[256];
  __shared__ int s_nact, s_bad, s_tsmall, s_tsingle, s_rhot;
  const int tid = threadIdx.x, E = A.n_experts;
  const int64_t S = A.t * A.topk;
  for (int e = tid; e < E; e += 256) s_cnt[e] = 0;
  if (tid == 0) {
    s_bad = 0;
    s_nact = 0;
    s_tsmall = 0x7fffffff;
    s_tsingle = 0x7fffffff;
    s_rhot = 0x7fffffff;
  }
  __syncthreads();
  // The slots' expert ids, kSB per thread at a time, all requested before any is used
  // (one round trip per batch rather than one per slot); a step of at most 256 * kSB
  // slots keeps its one batch in registers for the placement pass at the end.
  constexpr int kSB = 16;
  int ev[kSB];
  const auto load_ids = [&](int64_t s0) {
#pragma unroll
    for (int i = 0; i < kSB; ++i) ev[i] = A.topk_idx[min(s0 + tid + 256 * i, S - 1)];
    __builtin_amdgcn_sched_barrier(0);
  };
  for (int64_t s0 = 0; s0 < S; s0 += 256 * kSB) {
    load_ids(s0);
#pragma unroll
    for (int i = 0; i < kSB; ++i) {
      if (s0 + tid + 256 * i >= S) continue;
      const int e = ev[i];
      if (e >= 0 && e < E) atomicAdd(&s_cnt[e], 1);
      else s_bad = 1;
    }
  }
  __syncthreads();
  // Rank the active experts. With more than one token per step, hottest first (count
  // descending, id ascending): the work queues below hand out tasks in rank order, so
  // the longest tasks start first, one per workgroup. One token (or more experts or
  // slots than the key below holds): id order. The order only schedules work; no
  // output depends on it.
  const bool by_count = A.t > 1 && E <= 1024 && S < ((int64_t)1 << 19);
  if (by_count) {
    // key = count above (2047 - id): distinct, and larger exactly for an earlier rank;
    // 0 for an inactive expert. A rank counts the larger keys, four per broadcast LDS
    // read (a loop of dependent single reads costs an LDS round trip per expert).
    const int E4 = (E + 3) & ~3;
    for (int e = tid; e < E4; e += 256) {
      const int c = e < E ? s_cnt[e] : 0;
      s_base[e] = c > 0 ? (c << 11) | (2047 - e) : 0;
      if (c > 0) atomicAdd(&s_nact, 1);
    }
    __syncthreads();
    const int4* k4 = reinterpret_cast<const int4*>(s_base);
    for (int e = tid; e < E; e += 256) {
      const int k = s_base[e];
      if (k == 0) continue;
      int r = 0;
#pragma unroll 8
      for (int i = 0; i < E4 / 4; ++i) {
        const int4 v = k4[i];
        r += (v.x > k) + (v.y > k) + (v.z > k) + (v.w > k);
      }
      s_ebr[r] = e;
    }
  } else {
    // an expert's rank is the number of active experts below it: a scan of the active
    // flags over contiguous id ranges
    const int per = (E + 255) / 256, e0 = min(E, tid * per), e1 = min(E, e0 + per);
    int na = 0;
    for (int e = e0; e < e1; ++e) na += s_cnt[e] > 0;
    s_scan[tid] = na;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {
      const int v = tid >= off ? s_scan[tid - off] : 0;
      __syncthreads();
      s_scan[tid] += v;
      __syncthreads();
    }
    int r = s_scan[tid] - na;
    for (int e = e0; e < e1; ++e)
      if (s_cnt[e] > 0) s_ebr[r++] = e;
    if (tid == 255) s_nact = s_scan[255];
  }
  __syncthreads();
  const int n_active = s_nact;
  // exclusive scan of the slot counts in rank order, contiguous ranks per thread
  const int per = (n_active + 255) / 256;
  const int r0 = min(n_active, tid * per), r1 = min(n_active, r0 + per);
  // (and of the token tiles: kMT-token tiles of every expert for the MFMA path; on the
  // mixed path (t32) instead the kMTs-token tiles of the experts of more than hyb slots,
  // which its MFMA role takes, in the lists tile32_exp / tt32_off)
  const bool t32 = by_count && A.hyb > 0;
  const auto ntiles = [&](int c) { return t32 ? (c > A.hyb ? (c + kMTs - 1) / kMTs : 0) : (c + kMT - 1) / kMT; };
  int ns = 0, nt = 0;
  for (int r = r0; r < r1; ++r) {
    ns += s_cnt[s_ebr[r]];
    nt += ntiles(s_cnt[s_ebr[r]]);
  }
  s_scan[tid] = ns;
  s_scan2[tid] = nt;
  __syncthreads();
  for (int off = 1; off < 256; off <<= 1) {
    const int v = tid >= off ? s_scan[tid - off] : 0;
    const int v2 = tid >= off ? s_scan2[tid - off] : 0;
    __syncthreads();
    s_scan[tid] += v;
    s_scan2[tid] += v2;
    __syncthreads();
  }
  int pos = s_scan[tid] - ns, tpos = s_scan2[tid] - nt;
  for (int r = r0; r < r1; ++r) {
    const int e = s_ebr[r];
    // In count order the experts of at most kMTs slots form the tail of the tile list, the
    // experts of one kMT-token tile the tail of the first launch's tiles and, on the mixed
    // path, the experts of at most hyb slots the tail of the small-tile ones: the rank at
    // which the count first falls to a bound records itself and its first tile (one plain
    // store each, where an atomic minimum over the tail would queue on one LDS word).
    if (by_count) {
      const int c = s_cnt[e], cprev = r > 0 ? s_cnt[s_ebr[r - 1]] : 0x7fffffff;
      if (c <= kMTs && cprev > kMTs) s_tsmall = tpos;
      if (c <= kMT && cprev > kMT) s_tsingle = tpos;
      if (c <= A.hyb && cprev > A.hyb) s_rhot = r;
    }
    A.active[r] = e;
    A.act_off[r] = pos;
    s_base[e] = pos;  // key no longer needed: becomes the expert's slot cursor
    pos += s_cnt[e];
    const int n_t = ntiles(s_cnt[e]);
    int32_t* const tt = t32 ? A.tt32_off : A.tt_off;
    int32_t* const te = t32 ? A.tile32_exp : A.tile_exp;
    if (n_t > 0 || !t32) tt[r] = tpos;
    for (const int t1 = tpos + n_t; tpos < t1; ++tpos) te[tpos] = r;
  }
  __syncthreads();
  if (tid == 255) {
    const int n_valid = s_scan[255], n_tiles = s_scan2[255];
    const int t_small = min(s_tsmall, n_tiles);
    A.act_off[n_active] = n_valid;
    (t32 ? A.tt32_off : A.tt_off)[n_active] = n_tiles;
    A.ctrl[kNActive] = n_active;
    A.ctrl[kNValid] = n_valid;
    A.ctrl[kTasksGU] = n_active * A.tiles_gu;
    A.ctrl[kTasksDn] = n_active * A.tiles_dn;
    A.ctrl[kTasksMGU] = t_small * A.tiles_mgu;
    A.ctrl[kTasksMDn] = t_small * A.tiles_mdn;
    A.ctrl[kTSmall] = t_small;
    A.ctrl[kTSingle] = min(s_tsingle, t_small);
    A.ctrl[kTasksMGUs] = (n_tiles - t_small) * A.tiles_mgus;
    A.ctrl[kTasksMDns] = (n_tiles - t_small) * A.tiles_mdns;
    A.ctrl[kRSkip] = 0;
    if (A.hyb > 0) {
      // ranks 0 .. rhot - 1 (more than hyb slots) go to the MFMA role in kMTs-token tiles
      // (the list tile32_exp, n_tiles of them); the VALU role takes ranks rhot on. (Not
      // by count: no MFMA tiles, every rank on the VALU role.)
      const int rhot = t32 ? min(s_rhot, n_active) : 0;
      A.ctrl[kRSkip] = rhot;
      A.ctrl[kTasksGU] = (n_active - rhot) * A.tiles_gu;
      A.ctrl[kTasksDn] = (n_active - rhot) * A.tiles_dn;
      A.ctrl[kTasksMGUs] = t32 ? n_tiles * A.tiles_mgus : 0;
      A.ctrl[kTasksMDns] = t32 ? n_tiles * A.tiles_mdns : 0;
    }
    A.ctrl[kFlags] = s_bad ? 1 : 0;
  }
  __syncthreads();
  for (int64_t s0 = 0; s0 < S; s0 += 256 * kSB) {
    if (S > 256 * kSB) load_ids(s0);  // otherwise ev still holds the only batch
#pragma unroll
    for (int i = 0; i < kSB; ++i) {
      const int64_t s = s0 + tid + 256 * i;
      if (s >= S) continue;
      const int e = ev[i];
      if (e >= 0 && e < E) {
        const int p = atomicAdd(&s_base[e], 1);
        A.slot_list[p] = (int)s;
      } else {
        // an unrouted slot: its hidden row is defined (zero) so the requant stage reads
        // finite values; the combine skips the slot.
        float4* hp = reinterpret_cast<float4*>(A.h + s * A.inter);
        for (int c = 0; c < A.inter / 4; ++c) hp[c] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
    }
  }
}

// ---------------------------------------------------------------------------------
// Grouped decode on the VALU (a few tokens per expert): task = (active expert, row
// tile), tasks in rank order strided over the grid. Each wave owns RPW rows of every
// matrix of the projection (gate and up, or down), reads them once and keeps them in
// registers already unpacked to 16c bytes, then walks the expert's tokens NT at a time
// (the last ones singly). Loads are issued unconditionally from clamped addresses
// (a predicated load becomes a branch that waits for it), and a block that does not
// exist (ragged k) or a token past the list gets d = 0, which adds exactly nothing.
// ---------------------------------------------------------------------------------

// One group of NT tokens (list positions c0 .. c0 + NT - 1) as the lane needs it: their
// slots, their 32 activation codes per load, and the block scales of the lane's kept
// items (as loaded: the compute zeroes those past the list or past kb, so that no use of
// a loaded value sits among the loads). Positions past the list repeat the last one.
template <int NMAT, int NL, int RPW, int NT>
struct TbActs {
  static constexpr int KI = RowReduce<RPW * NT, NMAT>::KI;
  int slot[NT];
  int q[NT][NL][8];
  float d[KI][NL];
};

// sv: lane p holds the slot of list position p (p < 64); later positions from the list.
template <int NMAT, int NL, int RPW, int NT, bool RAGGED>
__device__ __forceinline__ void tb_acts_load(const MoeArgs& A, __amdgpu_buffer_rsrc_t qr, __amdgpu_buffer_rsrc_t dr,
                                             int K, int kb, int sv, int off, int cnt, int c0, int lane, int g, int cp,
                                             TbActs<NMAT, NL, RPW, NT>& T) {
  using RR = RowReduce<RPW * NT, NMAT>;
  int arow[NT];
#pragma unroll
  for (int tt = 0; tt < NT; ++tt) {
    const int p = min(c0 + tt, cnt - 1);
    T.slot[tt] = p < 64 ? __builtin_amdgcn_readlane(sv, p) : A.slot_list[off + p];
    arow[tt] = NMAT == 2 ? T.slot[tt] / A.topk : T.slot[tt];
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const uint32_t bc = (uint32_t)min(8 * i + g, kb - 1);
      const uint4 lo = buf_load16(qr, bc * 256u + (uint32_t)cp * 32u, (uint32_t)arow[tt] * (uint32_t)K, 0);
      const uint4 hi = buf_load16(qr, bc * 256u + (uint32_t)cp * 32u + 16u, (uint32_t)arow[tt] * (uint32_t)K, 0);
      T.q[tt][i][0] = (int)lo.x; T.q[tt][i][1] = (int)lo.y; T.q[tt][i][2] = (int)lo.z; T.q[tt][i][3] = (int)lo.w;
      T.q[tt][i][4] = (int)hi.x; T.q[tt][i][5] = (int)hi.y; T.q[tt][i][6] = (int)hi.z; T.q[tt][i][7] = (int)hi.w;
    }
  }
#pragma unroll
  for (int k = 0; k < RR::KI; ++k) {
    const int tt = RR::kept(k, lane) % NT;
    int ar = arow[0];
#pragma unroll
    for (int u = 1; u < NT; ++u) ar = tt == u ? arow[u] : ar;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const uint32_t bc = (uint32_t)min(8 * i + g, kb - 1);
      T.d[k][i] = __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(dr, ((uint32_t)ar * (uint32_t)kb + bc) * 4u, 0, 0));
    }
  }
}

// The token group against the wave's NMAT x RPW rows, whose codes the lane holds
// unpacked (wc[m * RPW + r][i]) with the scales of its own row (sl[m][i]: after the
// block butterfly a lane keeps items of one row, rev(lane bits) for RPW <= 8). Items are
// (row r, token tt) = r * NT + tt, each for the NMAT matrices.
template <int NMAT, int NL, int RPW, int NT, bool RAGGED>
__device__ __forceinline__ void tb_acts_compute(const MoeArgs& A, const int (&wc)[NMAT * RPW][NL][8],
                                                const float (&sl)[NMAT][NL], const TbActs<NMAT, NL, RPW, NT>& T, int N,
                                                int kb, int cnt, int c0, int row0, int lane) {
  using RR = RowReduce<RPW * NT, NMAT>;
  constexpr int KI = RR::KI;
  const int g = lane >> 3;
  float acc[KI * NMAT];
#pragma unroll
  for (int v = 0; v < KI * NMAT; ++v) acc[v] = 0.0f;
  // a kept item's block scale, zero for a token past the list or a block past kb
  float dk[KI][NL];
#pragma unroll
  for (int k = 0; k < KI; ++k) {
    const bool tv = c0 + RR::kept(k, lane) % NT < cnt;
#pragma unroll
    for (int i = 0; i < NL; ++i) dk[k][i] = (tv && (!RAGGED || 8 * i + g < kb)) ? T.d[k][i] : 0.0f;
  }
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    int p[RPW * NT * NMAT];
#pragma unroll
    for (int r = 0; r < RPW; ++r)
#pragma unroll
      for (int tt = 0; tt < NT; ++tt)
#pragma unroll
        for (int m = 0; m < NMAT; ++m) p[(r * NT + tt) * NMAT + m] = dot32x16(wc[m * RPW + r][i], T.q[tt][i]);
    RR::block_sums(p);
    // debug stage dump: the exact block sums of the kept items, one lane per item
    if ((NMAT == 2 ? A.dbg_gsum : A.dbg_dsum) != nullptr && RR::block_writer(lane) && 8 * i + g < kb) {
#pragma unroll
      for (int k = 0; k < KI; ++k) {
        const int it = RR::kept(k, lane), r = it / NT, tt = it % NT;
        int sv = T.slot[0];
#pragma unroll
        for (int u = 1; u < NT; ++u) sv = tt == u ? T.slot[u] : sv;
        if (row0 + r < N && c0 + tt < cnt) {
          const int64_t o = ((int64_t)sv * N + row0 + r) * kb + 8 * i + g;
          if constexpr (NMAT == 2) {
            A.dbg_gsum[o] = p[k * 2] >> 4;
            A.dbg_usum[o] = p[k * 2 + 1] >> 4;
          } else {
            A.dbg_dsum[o] = p[k] >> 4;
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < KI; ++k)
#pragma unroll
      for (int m = 0; m < NMAT; ++m)
        acc[k * NMAT + m] = fmaf(sl[m][i] * dk[k][i], (float)(p[k * NMAT + m] >> 4), acc[k * NMAT + m]);
  }
  RR::block_totals(acc);
  if (RR::writer(lane)) {
    const int it = RR::item(lane), r = it / NT, tt = it % NT;
    int sv = T.slot[0];
#pragma unroll
    for (int u = 1; u < NT; ++u) sv = tt == u ? T.slot[u] : sv;
    if (row0 + r < N && c0 + tt < cnt) {
      if constexpr (NMAT == 2) {
        const int64_t o = (int64_t)sv * A.inter + row0 + r;
        A.h[o] = silu_f32(acc[0]) * acc[1];
        if (A.dbg_g != nullptr) {
          A.dbg_g[o] = acc[0];
          A.dbg_u[o] = acc[1];
        }
      } else {
        A.yd[(int64_t)sv * A.hidden + row0 + r] = acc[0];
      }
    }
  }
}

// A task's scalars (its active expert's slot-list range and id) in one vector load:
// lane 0 gets the range's start, lane 1 its end, lane 2 the expert id. Kept in a vector
// register and read out lane by lane only where used, so that a fetch issued one task
// ahead is not waited for at once.
// (on the mixed path the VALU role's task ranks start at rskip, past the MFMA role's)
__device__ __forceinline__ int tb_task_fetch(const MoeArgs& A, int task, int tiles, int lane, int rskip) {
  const int a = task / tiles + rskip;
  return *(lane == 2 ? A.active + a : A.act_off + a + (lane & 1));
}
struct TbTask {
  int64_t e;
  int off, cnt, tile;
};
__device__ __forceinline__ TbTask tb_task(int v, int task, int tiles) {
  const int off = __builtin_amdgcn_readlane(v, 0);
  return {(int64_t)__builtin_amdgcn_readlane(v, 2), off, __builtin_amdgcn_readlane(v, 1) - off, task % tiles};
}

// NMAT == 2: h[slot][row] = SiLU(Wg[e] xq[token]) * (Wu[e] xq[token]);
// NMAT == 1: yd[slot][row] = Wd[e] hq[slot].
// Per task, in issue order: the wave's weight rows, then the first token group's
// activations (their slots, the expert's first 64, one per lane, came in during the task
// before), so that their round trip overlaps the weights' (most tasks have a single
// group); then the next task's slots; further groups load and compute in turn (the last
// one possibly part-empty).
// `bid` of `nblk`: the workgroup's index among those that run this role (the whole grid
// for k_tb, the workgroups past the MFMA ones in k_mixed).
template <int NMAT, int NL, int RPW, int NT, int NTL, int WAVES, bool RAGGED>
__device__ __forceinline__ void tb_run(const MoeArgs& A, int bid, int nblk) {
  static_assert(RPW <= 8 && (RPW & (RPW - 1)) == 0, "RPW: a power of two <= 8");
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 3, cp = lane & 7;
  const int K = NMAT == 2 ? A.hidden : A.inter;
  const int N = NMAT == 2 ? A.inter : A.hidden;
  const int kb = K / 256;
  const int tiles = NMAT == 2 ? A.tiles_gu : A.tiles_dn;
  const int n_tasks = A.ctrl[NMAT == 2 ? kTasksGU : kTasksDn];
  const int rskip = A.ctrl[kRSkip];
  const uint32_t arows = (uint32_t)(NMAT == 2 ? A.t : A.t * A.topk);
  const __amdgpu_buffer_rsrc_t qr = make_rsrc(NMAT == 2 ? A.xq : A.hq, arows * (uint32_t)K);
  const __amdgpu_buffer_rsrc_t dr = make_rsrc(NMAT == 2 ? A.xd : A.hd, arows * (uint32_t)kb * 4u);
  const int lr = rev_bits<clog2(RPW)>(lane & (RPW - 1));  // the lane's row after the block butterfly
  int task = bid;
  if (task >= n_tasks) return;
  // A task's scalars and slot list are fetched while the task before it runs (at its own
  // start each would be another round trip ahead of the weight loads).
  int tv = tb_task_fetch(A, task, tiles, lane, rskip);
  int sv;
  {
    const TbTask t0 = tb_task(tv, task, tiles);
    sv = A.slot_list[t0.off + min(lane, t0.cnt - 1)];
  }
  for (; task < n_tasks; task += nblk) {
    const TbTask cur = tb_task(tv, task, tiles);
    const int task_next = min(task + nblk, n_tasks - 1);
    const int tv_next = tb_task_fetch(A, task_next, tiles, lane, rskip);
    const int64_t e = cur.e;
    const int off = cur.off, cnt = cur.cnt;
    // rows past N (a ragged last tile) load the last row and write nothing
    const int row0 = (cur.tile * WAVES + wv) * RPW;
    constexpr int NF = NT > 1 ? NT : 1;  // the first group's width
    TbActs<NMAT, NL, RPW, NF> first;
    int wc[NMAT * RPW][NL][8];
    float sl[NMAT][NL];
    int sv_next;
    {
      uint4 raw[NMAT * RPW][NL];
      uint16_t sr[NMAT][NL];
#pragma unroll
      for (int m = 0; m < NMAT; ++m) {
        const int p = NMAT == 2 ? m : 2;
        const MatRsrc mr = mat_rsrc(A.codes[p] + e * A.stride_codes[p], A.scales[p] + e * A.stride_scales[p], N, kb);
#pragma unroll
        for (int r = 0; r < RPW; ++r) {
          const uint32_t srow = (uint32_t)min(row0 + r, N - 1) * (uint32_t)kb;
#pragma unroll
          for (int i = 0; i < NL; ++i) {
            const uint32_t bc = (uint32_t)min(8 * i + g, kb - 1);
            raw[m * RPW + r][i] = buf_load16(mr.codes, bc * 128u + (uint32_t)cp * 16u, srow * 128u);
          }
        }
        // the lane's row (lane-varying, so in the vector offset)
        const uint32_t lrow = (uint32_t)min(row0 + lr, N - 1) * (uint32_t)kb;
#pragma unroll
        for (int i = 0; i < NL; ++i) sr[m][i] = buf_load_u16(mr.scales, (lrow + (uint32_t)min(8 * i + g, kb - 1)) * 2u, 0);
      }
      tb_acts_load<NMAT, NL, RPW, NF, RAGGED>(A, qr, dr, K, kb, sv, off, cnt, 0, lane, g, cp, first);
      // the next task's slots, after this task's loads and ahead of the wait for them
      __builtin_amdgcn_sched_barrier(0);
      {
        const TbTask nxt = tb_task(tv_next, task_next, tiles);
        sv_next = A.slot_list[nxt.off + min(lane, nxt.cnt - 1)];
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int v = 0; v < NMAT * RPW; ++v)
#pragma unroll
        for (int i = 0; i < NL; ++i) unpack16c(raw[v][i], wc[v][i]);
#pragma unroll
      for (int m = 0; m < NMAT; ++m)
#pragma unroll
        for (int i = 0; i < NL; ++i) sl[m][i] = f16_bits_to_f32(sr[m][i]);
    }
    tb_acts_compute<NMAT, NL, RPW, NF, RAGGED>(A, wc, sl, first, N, kb, cnt, 0, row0, lane);
    for (int c0 = NF; c0 < cnt; c0 += NTL) {
      TbActs<NMAT, NL, RPW, NTL> grp;
      tb_acts_load<NMAT, NL, RPW, NTL, RAGGED>(A, qr, dr, K, kb, sv, off, cnt, c0, lane, g, cp, grp);
      tb_acts_compute<NMAT, NL, RPW, NTL, RAGGED>(A, wc, sl, grp, N, kb, cnt, c0, row0, lane);
    }
    tv = tv_next;
    sv = sv_next;
  }
}

template <int NMAT, int NL, int RPW, int NT, int NTL, int WAVES, bool RAGGED>
__global__ __launch_bounds__(WAVES * 64) void k_tb(MoeArgs A) {
  tb_run<NMAT, NL, RPW, NT, NTL, WAVES, RAGGED>(A, blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------------
// requant and combine
// ---------------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_moe_requant(MoeArgs A, int64_t nblocks) {
  quantize_wave_blocks(A.h, nblocks, (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6), A.hq, A.hd, A.hb);
}

__global__ __launch_bounds__(256) void k_moe_combine(MoeArgs A, float* __restrict__ out) {
  const int64_t H4 = A.hidden / 4;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= A.t * H4) return;
  const int64_t tok = i / H4, c4 = i - tok * H4;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  // eight slots at a time: their ids, weights and rows load together (one round trip,
  // not one per slot; positions past topk reload the last slot and are skipped), then
  // the sum goes on in ascending j, skipping unrouted slots (their rows are never written)
  constexpr int kJ = 8;
  for (int j0 = 0; j0 < A.topk; j0 += kJ) {
    int e[kJ];
    float w[kJ];
    float4 v[kJ];
#pragma unroll
    for (int u = 0; u < kJ; ++u) {
      const int64_t s = tok * A.topk + min(j0 + u, A.topk - 1);
      e[u] = A.topk_idx[s];
      w[u] = A.topk_w[s];
      v[u] = reinterpret_cast<const float4*>(A.yd + s * A.hidden)[c4];
    }
#pragma unroll
    for (int u = 0; u < kJ; ++u) {
      if (j0 + u >= A.topk || e[u] < 0 || e[u] >= A.n_experts) continue;
      acc.x = fmaf(w[u], v[u].x, acc.x);
      acc.y = fmaf(w[u], v[u].y, acc.y);
      acc.z = fmaf(w[u], v[u].z, acc.z);
      acc.w = fmaf(w[u], v[u].w, acc.w);
    }
  }
  reinterpret_cast<float4*>(out)[i] = acc;
}

// ---------------------------------------------------------------------------------
// Many tokens per expert (prefill-sized groups): the per-expert contraction is a dense
// int8 GEMM, run on v_mfma_i32_16x16x64_i8. A workgroup of kMWaves waves owns one task:
// kMT tokens of one active expert x kMN weight rows (x2 matrices for gate/up); wave w
// owns rows 16w .. 16w + 15 of the tile for all kMT tokens. The block scales of the
// tile's tokens go to LDS once per task. Per 256-column block:
//  - the token tile's codes (kMT x 256 bytes) travel by direct-to-LDS loads into a ring
//    of kMStages stages, kMStages - 1 blocks ahead of the compute; 16-byte column c of
//    row r sits at column c ^ (r & 15), so the 16 lanes that read one operand column of
//    16 rows hit distinct banks;
//  - each wave loads its 16 rows' nibbles kMStages - 1 blocks ahead into registers,
//    row-coalesced (four neighbouring lanes read one 64-byte half of a row block: with
//    one row per lane, each load would fetch sixteen 16-byte pieces of different rows,
//    and the loads issue far slower), rewrites them through its own LDS area into MFMA
//    lane order and unpacks them to 16c bytes as the B operands (lane: row l & 15, chunk
//    4t + (l >> 4), half h gives MFMA (t, h); the A operand takes the same 16 columns of
//    the token's codes, so every product pairs matching columns);
//  - four MFMAs per 16x16 output tile accumulate sum (16c)*q = 16 * isum exactly (two
//    sub-tiles at a time, so that 2 * NMAT independent chains interleave), and one
//    fp32 multiply-add per output applies (f32(s) / 16) * d to it; pairs of 16-token
//    sub-tiles past the expert's last token are skipped, and so are their token loads.
// Tasks run hottest expert first, row tiles innermost: the workgroups running together
// share a token tile through L2, and the tasks of one weight tile run RT tasks apart.
// ---------------------------------------------------------------------------------

typedef int v4i __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void* lds_ptr;

// A wave-uniform read of data that no kernel still running writes (here: the prologue's
// control data), through the constant address space, so that it is a scalar load.
template <typename T>
__device__ __forceinline__ T ld_uniform(const T* p) {
  return *reinterpret_cast<const __attribute__((address_space(4))) T*>(reinterpret_cast<uintptr_t>(p));
}

__device__ __forceinline__ v4i lds_v4i(const int8_t* p) {
  const int4 v = *reinterpret_cast<const int4*>(p);
  return v4i{v.x, v.y, v.z, v.w};
}

// s_waitcnt with only the vector-memory count constrained (gfx9 encoding: vmcnt in bits
// 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt out of range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// One block's weights for one wave, per matrix: two 16-byte code chunks per lane as
// loaded (row-coalesced: load c gives lane l chunk l & 7 of the wave's row 8c + (l >> 3),
// so eight neighbouring lanes read one row's whole 128-byte block, one cache line), and
// the scale of the lane's MFMA row l & 15.
template <int NMAT>
struct MfmaB {
  uint4 w[NMAT][2];
  uint32_t s[NMAT];  // f16 bits, zero-extended
};

// A buffer offset past every resource's num_records (all below 2^31 bytes): a load there
// returns zeros without a memory access but still counts as an issued load, so refills
// that are not needed keep every wave's count of loads in flight the same.
constexpr uint32_t kOob = 0x80000000u;

// Block b's weights for one wave whose 16 rows start at row0 (wrow: the lane's MFMA row;
// b >= kb: out of range, no memory access). Cached loads: a hot expert's rows are read
// again by its other token tiles.
template <int NMAT>
__device__ __forceinline__ void mfma_b_fetch(MfmaB<NMAT>& B, const MatRsrc (&mr)[NMAT], int row0, int wrow, int kb,
                                             int lane, int b) {
  const bool live = b < kb;
  // (scales first: the compiler's own wait before the first reader of the last load of
  // the group, a code chunk that the LDS store above takes after the step's wait, stays
  // partial)
#pragma unroll
  for (int m = 0; m < NMAT; ++m) B.s[m] = buf_load_u16(mr[m].scales, live ? (uint32_t)((wrow * kb + b) * 2) : kOob, 0);
#pragma unroll
  for (int m = 0; m < NMAT; ++m) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
      B.w[m][c] = buf_load16(mr[m].codes,
                             live ? (uint32_t)(((row0 + 8 * c + (lane >> 3)) * kb + b) * 128 + (lane & 7) * 16) : kOob,
                             0, 0);
  }
}

// Piece j of block b of the token tile into one ring stage: 1 KB of codes, rows
// 4 (4w + j) .. + 3 (ao: the lane's byte offset from q for this piece at block 0). A piece
// that is not needed (a sub-tile the task does not compute, or b >= kb) reads the first
// 16 bytes of the activations in every lane: one cache line instead of 1 KB.
template <int PW>
__device__ __forceinline__ void mfma_a_dma(int8_t* sa, const int8_t* q, uint32_t ao, bool live, int b, int kb, int wv,
                                           int j) {
  const uint32_t o = live && b < kb ? ao + (uint32_t)b * 256u : 0u;
  __builtin_amdgcn_global_load_lds((const void*)(q + o), (lds_ptr)(sa + (wv * PW + j) * 1024), 16, 0, 0);
}

// Per block and wave: PW code pieces and three loads per matrix.
template <int NMAT, int PW>
constexpr int kMfmaLoadsPerBlock = PW + 3 * NMAT;

// NMAT 2: gate and up, h = SiLU(g) * u; 1: down, y per slot. MT tokens x 16 WAVES rows per
// task; SMALL: the launch for the tail of the tile list (experts of at most kMTs slots).
// DBG: the instance that also writes the debug stage dumps (launched only when they are
// requested, so that the production instances carry no dump code or its registers).
// DN2: the down projection with two 16-row tiles of the matrix per wave, run as the two
// "matrices" of the NMAT = 2 path (the second's resource starts 16 rows on), so that each
// token operand read from LDS feeds two MFMAs, as in gate/up.
// T32: the mixed path's MFMA role, whose tasks walk the kMTs-token tile list (tile32_exp,
// every tile of the experts of more than hyb slots) instead of the kMT-token one.
// `bid` of `nblk` as in tb_run (the whole grid for k_moe_mfma, the first workgroups of
// k_mixed).
template <int NMAT, int MT, int WAVES, bool SMALL, bool DBG, bool DN2, bool T32>
__device__ __forceinline__ void mfma_run(const MoeArgs& A, int bid, int nblk) {
  static_assert(!DN2 || NMAT == 2, "DN2 runs two row tiles as two matrices");
  static_assert(!T32 || (SMALL && MT == kMTs), "the kMTs-token tile list feeds the small-tile instance");
  constexpr bool GU = NMAT == 2 && !DN2;  // the gate/up projection
  constexpr int RW = DN2 ? 32 : 16;       // weight rows per wave
  constexpr int MN = RW * WAVES;          // weight rows per task
  constexpr int PW = MT / (4 * WAVES);  // 1 KB token pieces (4 token rows) per wave and block
  // one variable per ring stage, and stages chosen at compile time, so that the compiler
  // can tell a stage being filled from the one being read and does not wait for the fill
  __shared__ __attribute__((aligned(16))) int8_t s_a0[MT * 256], s_a1[MT * 256], s_a2[MT * 256];
  // [block][token], rows padded by 4 floats: the fill below (consecutive lanes take
  // consecutive blocks of one token) then writes distinct banks at 16 blocks
  constexpr int DS = MT + 4;
  __shared__ __attribute__((aligned(16))) float s_dall[(kMaxK / 256) * DS];
  __shared__ int s_slot[MT];
  // per wave: one matrix's block of its 16 rows (2 KB), the row-coalesced loads rewritten
  // in MFMA lane order; chunk x of row r at position x ^ ((r >> 1) & 7) of the row, so that
  // eight lanes writing one row, and eight lanes reading one chunk of eight rows, fall in
  // distinct banks
  __shared__ __attribute__((aligned(16))) uint8_t s_bt[WAVES * 2048];
  static_assert(MT % 32 == 0 && PW >= 2 && PW % 2 == 0 && 4 * PW * WAVES == MT && kMStages == 3, "tile geometry");
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, g = lane >> 4;
  const int K = GU ? A.hidden : A.inter;
  const int N = GU ? A.inter : A.hidden;
  const int kb = K / 256;
  const int RT = SMALL ? (GU ? A.tiles_mgus : A.tiles_mdns) : (GU ? A.tiles_mgu : A.tiles_mdn);
  const int n_tasks = ld_uniform(A.ctrl + (SMALL ? (GU ? kTasksMGUs : kTasksMDns) : (GU ? kTasksMGU : kTasksMDn)));
  const int tile0 = SMALL && !T32 ? ld_uniform(A.ctrl + kTSmall) : 0;
  const int8_t* qsrc = GU ? A.xq : A.hq;
  const float* dsrc = GU ? A.xd : A.hd;
  // Tiles before t1 (experts of several tiles): task = tile * RT + rtile, so one row tile
  // of all of an expert's token tiles runs on one XCD (the grid and RT are multiples of
  // 8, and workgroups go to the XCDs in turn) and its weights are fetched once. From t1
  // on every expert has one tile; in whole rounds of 8 such tiles, all row tiles of a
  // token tile run on one XCD, so that its token rows are fetched into one L2 only.
  const int t1 = SMALL ? tile0 : ld_uniform(A.ctrl + kTSingle);
  const int n_single = (SMALL ? n_tasks / RT : ld_uniform(A.ctrl + kTSmall) - t1);
  const int base1 = (t1 - tile0) * RT, full1 = (n_single / 8) * 8 * RT;
  for (int task = bid; task < n_tasks; task += nblk) {
    // the control data was written by the prologue kernel, so it is read through the
    // scalar cache (not queued behind this compute unit's vector loads)
    int tile, rtile;
    const int k = task - base1;
    if (k < 0 || k >= full1) {
      tile = tile0 + task / RT;
      rtile = task - (task / RT) * RT;
    } else {
      const int x = k & 7, i = k >> 3;  // XCD x's i-th task
      tile = t1 + x + 8 * (i / RT);
      rtile = i - (i / RT) * RT;
    }
    const int a = ld_uniform((T32 ? A.tile32_exp : A.tile_exp) + tile);
    const int ttile = tile - ld_uniform((T32 ? A.tt32_off : A.tt_off) + a);
    const int64_t e = ld_uniform(A.active + a);
    const int off = ld_uniform(A.act_off + a), cnt = ld_uniform(A.act_off + a + 1) - off;
    // (SMALL: one tile, ttile 0, except on the T32 list)
    const int m0 = ttile * (T32 ? MT : kMT), nvalid = min(MT, cnt - m0);
    const int nsub = (nvalid + 15) / 16;  // 16-token sub-tiles holding valid tokens
    const int ncomp = 2 * ((nsub + 1) / 2);  // sub-tiles computed (in pairs)
    const int row0 = rtile * MN + wv * RW;  // N is a multiple of 256: all the wave's rows exist
    const int wrow = row0 + li;
    MatRsrc mr[NMAT];
#pragma unroll
    for (int m = 0; m < NMAT; ++m) {
      const int p = GU ? m : 2;
      // (DN2: the second tile's resource starts 16 rows on)
      const int64_t r16 = DN2 ? 16 * m : 0;
      mr[m] = mat_rsrc(A.codes[p] + e * A.stride_codes[p] + r16 * kb * 128, A.scales[p] + e * A.stride_scales[p] + r16 * kb,
                       N - (int)r16, kb);
    }
    __syncthreads();  // the previous task is done with the ring, s_slot and s_dall
    // Set-up in the order that keeps its round trips short: the slot list first (the token
    // side waits on it), then the weights of blocks 0 and 1, which need only the expert and
    // the row tile and so travel while the token side is set up; then, from the slots, the
    // token pieces of blocks 0 and 1 and the tile's block scales. Loads complete in issue
    // order, so each wait below covers exactly what precedes it.
    int my_slot = 0;
    if (threadIdx.x < MT) my_slot = A.slot_list[off + m0 + min((int)threadIdx.x, nvalid - 1)];
    __builtin_amdgcn_sched_barrier(0);
    // blocks 0 and 1 in flight; then per block b (block b's loads are in, block b + 1's may
    // not be): block b's weights through LDS into MFMA order, block b + 2's weights issued
    // into the registers just emptied, barrier (every wave's piece of block b is in LDS,
    // and stage (b + 2) % 3 is no longer read), block b + 2's pieces issued, block b
    // computed, then the wait for block b + 1 (loads complete in issue order).
    // Block b uses stage b % 3 and weight registers b % 2: the loop runs six blocks a turn.
    MfmaB<NMAT> B0, B1;
    mfma_b_fetch<NMAT>(B0, mr, row0, wrow, kb, lane, 0);
    __builtin_amdgcn_sched_barrier(0);
    mfma_b_fetch<NMAT>(B1, mr, row0, wrow, kb, lane, 1);
    __builtin_amdgcn_sched_barrier(0);
    if (threadIdx.x < MT) s_slot[threadIdx.x] = my_slot;
    __syncthreads();
    // the lane's direct-to-LDS sources: piece j covers rows 4 (PW w + j) .. + 3, the lane
    // row 4 (PW w + j) + (l >> 4) at stored column l & 15, i.e. source column (l & 15) ^ (r & 15);
    // wave w fills rows 4 PW w .. 4 PW (w + 1) - 1, so a wave past the computed sub-tiles loads nothing
    uint32_t ap[PW];  // (activations address below 2^31 bytes)
#pragma unroll
    for (int j = 0; j < PW; ++j) {
      const int r = (wv * PW + j) * 4 + (lane >> 4);
      const int sl = s_slot[r];
      const uint32_t arow = GU ? (uint32_t)(sl / A.topk) : (uint32_t)sl;
      ap[j] = arow * (uint32_t)K + (uint32_t)(((lane & 15) ^ (r & 15)) * 16);
    }
    const bool alive = 4 * PW * wv < 16 * ncomp;
#pragma unroll
    for (int j = 0; j < PW; ++j) mfma_a_dma<PW>(s_a0, qsrc, ap[j], alive, 0, kb, wv, j);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int j = 0; j < PW; ++j) mfma_a_dma<PW>(s_a1, qsrc, ap[j], alive, 1, kb, wv, j);
    __builtin_amdgcn_sched_barrier(0);
    // every block scale of the tile's computed tokens, once per task
    for (int i = threadIdx.x; i < 16 * ncomp * kb; i += WAVES * 64) {
      const int t = i / kb, b = i - t * kb, sl = s_slot[t];
      s_dall[b * DS + t] = dsrc[(GU ? (int64_t)(sl / A.topk) : (int64_t)sl) * kb + b];
    }
    __syncthreads();
    float acc[MT / 16][NMAT][4];
#pragma unroll
    for (int mt = 0; mt < MT / 16; ++mt)
#pragma unroll
      for (int m = 0; m < NMAT; ++m)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[mt][m][v] = 0.0f;
    // (every load above has completed: the block scales were loaded last)
    const auto step = [&](int b, auto stage_c, MfmaB<NMAT>& Bs) {
      constexpr int ST = decltype(stage_c)::value, NS = (ST + 2) % 3;
      const int8_t* const sa = ST == 0 ? s_a0 : (ST == 1 ? s_a1 : s_a2);
      int8_t* const na = NS == 0 ? s_a0 : (NS == 1 ? s_a1 : s_a2);
      const float* const sd = s_dall + b * DS;
      float sf[NMAT];
      v4i bop[NMAT][2][2];
      uint8_t* const bt = s_bt + wv * 2048;
#pragma unroll
      for (int m = 0; m < NMAT; ++m) {
        // the MFMA sums 16c * q = 16 isum; dividing the f16 scale by 16 is exact
        sf[m] = f16_bits_to_f32((uint16_t)Bs.s[m]) * 0.0625f;
        // through the wave's own LDS areas into MFMA order: lane (li, g) takes chunks g and
        // 4 + g of row li (LDS accesses of one wave complete in issue order, so the reads
        // see the writes; the fences keep the compiler's order)
        const int wr = lane >> 3;  // (row wr of the first load, 8 + wr of the second)
        *reinterpret_cast<uint4*>(bt + wr * 128 + (((lane & 7) ^ ((wr >> 1) & 7)) * 16)) = Bs.w[m][0];
        *reinterpret_cast<uint4*>(bt + (8 + wr) * 128 + (((lane & 7) ^ (((8 + wr) >> 1) & 7)) * 16)) = Bs.w[m][1];
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_wave_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        const int rs = (li >> 1) & 7;
        uint4 wt[2];
        wt[0] = *reinterpret_cast<const uint4*>(bt + li * 128 + ((g ^ rs) * 16));
        wt[1] = *reinterpret_cast<const uint4*>(bt + li * 128 + (((4 + g) ^ rs) * 16));
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
        __builtin_amdgcn_wave_barrier();
        __atomic_signal_fence(__ATOMIC_SEQ_CST);
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const uint4 w = wt[c];
          bop[m][c][0] = v4i{lo16c(w.x), lo16c(w.y), lo16c(w.z), lo16c(w.w)};
          bop[m][c][1] = v4i{hi16c(w.x), hi16c(w.y), hi16c(w.z), hi16c(w.w)};
        }
      }
      // block b + 2's weights into the registers emptied above (past the last block: out of
      // range, no memory access)
      mfma_b_fetch<NMAT>(Bs, mr, row0, wrow, kb, lane, b + 2);
      // A bare barrier: __syncthreads' release fence would also wait for the loads in
      // flight for the blocks ahead. The wait above covers this wave's part of block b;
      // its LDS reads of the previous block were consumed (waited for) by its MFMAs; the
      // signal fences keep the compiler from moving memory accesses across the barrier.
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_barrier();
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      // block b + 2 is issued among the sub-tiles' MFMAs, so that the eight waves' loads
      // do not queue up at once; unconditional, so that every path has the same loads in
      // flight (past the last block: out-of-range loads, no memory access)
      const int nb = b + 2;
      // sub-tiles in pairs: one straight-line stretch holds 2 * NMAT independent MFMA
      // chains, so one chain's epilogue overlaps the others' MFMAs (a pair whose second
      // sub-tile holds no valid token computes it anyway: its rows repeat the last valid
      // token and are not stored)
      // the operands of sub-tile pair mp (A codes of its 32 token rows, their block scales)
      const auto read_pair = [&](int mp, v4i (&aop)[2][2][2], float4 (&d4)[2]) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const int mt = 2 * mp + q;
          const int8_t* arow_lds = sa + (mt * 16 + li) * 256;
#pragma unroll
          for (int c = 0; c < 2; ++c)
#pragma unroll
            for (int h = 0; h < 2; ++h) aop[q][c][h] = lds_v4i(arow_lds + (((2 * (4 * c + g) + h) ^ li) * 16));
          d4[q] = *reinterpret_cast<const float4*>(&sd[mt * 16 + 4 * g]);
        }
      };
      // the next pair's operands are read from LDS right after the current pair's MFMAs
      // are issued (into the same registers), so their LDS latency overlaps the current
      // pair's epilogue
      v4i aop[2][2][2];
      float4 d4[2], d4n[2];
      read_pair(0, aop, d4);
#pragma unroll
      for (int mp = 0; mp < MT / 32; ++mp) {
        if (mp < PW / 2) {
          mfma_a_dma<PW>(na, qsrc, ap[2 * mp], alive, nb, kb, wv, 2 * mp);
          mfma_a_dma<PW>(na, qsrc, ap[2 * mp + 1], alive, nb, kb, wv, 2 * mp + 1);
        }
        if (2 * mp >= nsub) continue;  // no valid token in this pair
        v4i C[2][NMAT];
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int m = 0; m < NMAT; ++m) C[q][m] = v4i{0, 0, 0, 0};
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int q = 0; q < 2; ++q)
#pragma unroll
              for (int m = 0; m < NMAT; ++m)
                C[q][m] = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop[q][c][h], bop[m][c][h], C[q][m], 0, 0, 0);
        if (mp + 1 < MT / 32 && 2 * (mp + 1) < nsub) read_pair(mp + 1, aop, d4n);
        // debug stage dump: C = 16 * isum of token row mt * 16 + 4g + v, weight row orow
        if (DBG && (GU ? A.dbg_gsum : A.dbg_dsum) != nullptr) {
          const int orow = rtile * MN + wv * RW + li;
#pragma unroll
          for (int q = 0; q < 2; ++q)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
              const int t = (2 * mp + q) * 16 + 4 * g + v;
              if (t < nvalid && orow < N) {
                const int64_t o = ((int64_t)s_slot[t] * N + orow) * kb + b;
                if constexpr (GU) {
                  A.dbg_gsum[o] = C[q][0][v] >> 4;
                  A.dbg_usum[o] = C[q][1][v] >> 4;
                } else {
#pragma unroll
                  for (int m = 0; m < NMAT; ++m) A.dbg_dsum[o + (int64_t)16 * m * kb] = C[q][m][v] >> 4;
                }
              }
            }
        }
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int m = 0; m < NMAT; ++m) {
            // C = 16 * isum exactly (|C| < 2^21, so (float)C is exact too)
            const int mt = 2 * mp + q;
            acc[mt][m][0] = fmaf(sf[m] * d4[q].x, (float)C[q][m][0], acc[mt][m][0]);
            acc[mt][m][1] = fmaf(sf[m] * d4[q].y, (float)C[q][m][1], acc[mt][m][1]);
            acc[mt][m][2] = fmaf(sf[m] * d4[q].z, (float)C[q][m][2], acc[mt][m][2]);
            acc[mt][m][3] = fmaf(sf[m] * d4[q].w, (float)C[q][m][3], acc[mt][m][3]);
          }
        d4[0] = d4n[0];
        d4[1] = d4n[1];
      }
      // for the next step: block b + 1's loads are in (only block b + 2's may still be in
      // flight). Waiting here, at the end of the step, keeps every reader of those
      // registers after the wait.
      wait_vmcnt<kMfmaLoadsPerBlock<NMAT, PW>>();
    };
    using I0 = std::integral_constant<int, 0>;
    using I1 = std::integral_constant<int, 1>;
    using I2 = std::integral_constant<int, 2>;
    // (a step is reached only through the one before it, and the loop repeats only
    // after its sixth, so that the compiler sees the same loads in flight on every path)
    for (int b = 0;; b += 6) {
      step(b, I0{}, B0);
      if (b + 1 >= kb) break;
      step(b + 1, I1{}, B1);
      if (b + 2 >= kb) break;
      step(b + 2, I2{}, B0);
      if (b + 3 >= kb) break;
      step(b + 3, I0{}, B1);
      if (b + 4 >= kb) break;
      step(b + 4, I1{}, B0);
      if (b + 5 >= kb) break;
      step(b + 5, I2{}, B1);
      if (b + 6 >= kb) break;
    }
    // output: token tile row mt*16 + 4g + v, weight row orow (DN2: and orow + 16)
    const int orow = rtile * MN + wv * RW + li;
    if (orow < N) {
#pragma unroll
      for (int mt = 0; mt < MT / 16; ++mt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int t = mt * 16 + 4 * g + v;
          if (t < nvalid) {
            const int64_t slot = s_slot[t];
            if constexpr (GU) {
              A.h[slot * A.inter + orow] = silu_f32(acc[mt][0][v]) * acc[mt][1][v];
              if (DBG && A.dbg_g != nullptr) {
                A.dbg_g[slot * A.inter + orow] = acc[mt][0][v];
                A.dbg_u[slot * A.inter + orow] = acc[mt][1][v];
              }
            } else {
#pragma unroll
              for (int m = 0; m < NMAT; ++m) A.yd[slot * A.hidden + orow + 16 * m] = acc[mt][m][v];
            }
          }
        }
    }
  }
}

template <int NMAT, int MT, int WAVES, bool SMALL, bool DBG, bool DN2 = false, bool T32 = false>
// (the small-tile gate/up instance is held to the registers of three waves per SIMD)
__global__ __launch_bounds__(WAVES * 64) __attribute__((amdgpu_waves_per_eu(SMALL && NMAT == 2 ? 3 : 1))) void k_moe_mfma(
    MoeArgs A) {
  mfma_run<NMAT, MT, WAVES, SMALL, DBG, DN2, T32>(A, blockIdx.x, gridDim.x);
}

// The mixed path's projection in one launch: workgroups 0 .. n_mfma - 1 run the kMTs-token
// MFMA tasks of the experts of more than hyb and at most kMTs slots, the rest the grouped
// VALU tasks of the other experts (a uniform branch per workgroup; both roles are four
// waves). One launch instead of two streams joined by events: on this device each such
// edge between queues costs several microseconds of idle time. NMAT: as in k_tb (1 =
// down, whose MFMA role runs the two-tile DN2 form). The one-load down instance is held
// to the registers of three waves per SIMD (its LDS allows three workgroups per compute
// unit; without the bound the MFMA role's registers would leave it two).
template <int NMAT, int NL, int RPW, int NT, int NTL, bool RAGGED>
__global__ __launch_bounds__(kTbWaves * 64) __attribute__((amdgpu_waves_per_eu(NMAT == 1 && NL == 1 ? 3 : 1))) void
k_mixed(MoeArgs A, int n_mfma) {
  static_assert(kTbWaves == kMWavesS, "both roles run four-wave workgroups");
  if ((int)blockIdx.x < n_mfma)
    mfma_run<2, kMTs, kMWavesS, true, false, NMAT == 1, true>(A, blockIdx.x, n_mfma);
  else
    tb_run<NMAT, NL, RPW, NT, NTL, kTbWaves, RAGGED>(A, blockIdx.x - n_mfma, gridDim.x - n_mfma);
}

// ---------------------------------------------------------------------------------
// Single-token step (t == 1, topk <= 8): two kernels and no dispatch pass. Each slot
// is its own task (a duplicated expert is simply computed twice), so the expert comes
// straight from topk_idx; x is quantized once per workgroup into LDS while the weight
// loads are in flight; in the down kernel each slot's wave requantizes that slot's h in
// registers, and the workgroup folds the weighted combine in ascending slot order (the
// same fmaf chain as k_moe_combine).
// ---------------------------------------------------------------------------------

constexpr int kT1MaxTopk = 8;
constexpr int kT1MaxHq = 16384;  // topk * inter bytes of requantized hidden held in LDS

// A lane's slice of one token's quantized activations, from LDS: for load i, block
// b = 8i + g, chunk cp: 32 codes (blocks past the end of a row reread the last block;
// their scale d is taken as zero).
template <int NL>
__device__ __forceinline__ void lds_acts(const int8_t* s_q, int kb, int g, int cp, int (&q)[NL][8]) {
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int4* p = reinterpret_cast<const int4*>(s_q + min(8 * i + g, kb - 1) * 256 + cp * 32);
    const int4 lo = p[0], hi = p[1];
    q[i][0] = lo.x; q[i][1] = lo.y; q[i][2] = lo.z; q[i][3] = lo.w;
    q[i][4] = hi.x; q[i][5] = hi.y; q[i][6] = hi.z; q[i][7] = hi.w;
  }
}

// Row `row` (wave-uniform) of a matrix: the lane's NL 16-byte code chunks. Chunks past
// the row end reload the row's last block (their activations' scale is zero).
template <int NL>
__device__ __forceinline__ void load_lane_codes(const MatRsrc& m, int row, int kb, int g, int cp, uint4 (&w)[NL]) {
  const uint32_t srow = (uint32_t)row * (uint32_t)kb;
#pragma unroll
  for (int i = 0; i < NL; ++i)
    w[i] = buf_load16(m.codes, (uint32_t)min(8 * i + g, kb - 1) * 128u + (uint32_t)cp * 16u, srow * 128u);
}

// The lane's NL block scales of row `row` (per lane, so it goes in the vector offset: a
// lane-varying scalar offset would make the compiler loop over its distinct values).
template <int NL>
__device__ __forceinline__ void load_lane_scales(const MatRsrc& m, int row, int kb, int g, uint16_t (&s)[NL]) {
  const uint32_t srow = (uint32_t)row * (uint32_t)kb;
#pragma unroll
  for (int i = 0; i < NL; ++i) s[i] = buf_load_u16(m.scales, (srow + (uint32_t)min(8 * i + g, kb - 1)) * 2u, 0);
}

__device__ __forceinline__ int dot_chunk16(const uint4 w, const int (&a)[8]) {
  int c[8];
  unpack16c(w, c);
  return dot32x16(c, a);
}

// Layout of the single-token gate/up kernel's LDS: the quantized activations of the
// token, their block scales and code sums.
constexpr int kT1LdsQ = kMaxK;
constexpr int kT1LdsBytes = kT1LdsQ + 2 * (kT1LdsQ / 256) * 4;

struct T1Lds {
  int8_t* q;
  float* d;
  int* b;
  __device__ explicit T1Lds(uint8_t* raw)
      : q(reinterpret_cast<int8_t*>(raw)),
        d(reinterpret_cast<float*>(raw + kT1LdsQ)),
        b(reinterpret_cast<int*>(raw + kT1LdsQ + (kT1LdsQ / 256) * 4)) {}
};

// The activation quantizer on 16 lanes per 256-block (16 values a lane, lane (l & 15)
// holding values 16 (l & 15) .. + 15): the same rule as quantize_group32 (absmax by a
// butterfly over the 16 lanes, d = amax / 127 and inv = 127 / amax by IEEE division,
// q = rne(x * inv) by the 1.5 * 2^23 add), written to LDS at block blk; the block's d and
// code sum go to LDS from its first lane. Half the values a lane of the 8-lane form
// handles, so the block is ready sooner.
__device__ __forceinline__ void quantize16_to_lds(const float (&x)[16], int blk, int c16, int8_t* s_q, float* s_d,
                                                  int* s_b, bool store) {
#pragma clang fp contract(off)
  float a = 0.0f;
#pragma unroll
  for (int i = 0; i < 16; ++i) a = fmaxf(a, fabsf(x[i]));
  a = group_max_f32(a);
  a = fmaxf(a, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(a), kDppRowRor8, 0xf, 0xf, false)));
  int qw[4] = {0, 0, 0, 0};
  float d = 0.0f;
  int s = 0;
  if (a >= 0x1p-100f) {
    const float inv = 127.0f / a;
    d = a / 127.0f;
    constexpr float kMagic = 12582912.0f;  // 1.5 * 2^23
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      uint32_t b[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) b[k] = __float_as_uint(x[4 * m + k] * inv + kMagic);
      qw[m] = int(__builtin_amdgcn_perm(b[1], b[0], 0x0c0c0400u) | __builtin_amdgcn_perm(b[3], b[2], 0x04000c0cu));
      s = __builtin_amdgcn_sdot4(qw[m], 0x01010101, s, false);
    }
  }
  s = group_sum_i32(s);
  s += __builtin_amdgcn_update_dpp(0, s, kDppRowRor8, 0xf, 0xf, false);
  if (!store) return;
  *reinterpret_cast<int4*>(s_q + blk * 256 + c16 * 16) = make_int4(qw[0], qw[1], qw[2], qw[3]);
  if (c16 == 0) {
    s_d[blk] = d;
    s_b[blk] = s;
  }
}

// Gate/up of one single-token workgroup `wg`: WAVES waves, each owning RPW rows (a power
// of two) of gate and of up of one slot. x is quantized into LDS while the weight loads
// are in flight; per load, one integer butterfly forms the exact block sums, and the
// lanes that keep row rev(lane bits) apply the block scales; an fp32 butterfly over the
// blocks leaves each row's (g, u) in one lane, which writes h = SiLU(g) * u.
// `stage`: this workgroup also stores the quantized x and the status word.
template <int NL, int RPW, int WAVES, bool RAGGED>
__device__ __forceinline__ void t1_gateup_wg(const float* __restrict__ x, const MoeArgs& A, int wg, bool stage,
                                             T1Lds s) {
  static_assert(RPW == 1 || RPW == 2 || RPW == 4 || RPW == 8, "RPW must be a power of two <= 8");
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 3, cp = lane & 7;
  const int kb = A.hidden / 256, I = A.inter;
  const int j = wg / A.tiles_gu, tile = wg - j * A.tiles_gu;
  const int e = A.topk_idx[j];
  const bool valid = e >= 0 && e < A.n_experts;
  const int64_t ec = valid ? e : 0;
  const int row0 = (tile * WAVES + wv) * RPW;

  // x first (its wait must not queue behind the weights), then every weight load; a
  // workgroup quantizes x with 16 lanes per block: block 4 w + (l >> 4) of wave w, values
  // 16 (l & 15) .. + 15
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, (uint32_t)A.hidden * 4u);
  const int xb = wv * 4 + (lane >> 4), c16 = lane & 15;
  float v[16];
  const bool xw = wv * 4 < kb;  // wave-uniform: the wave has blocks of x to quantize
  if (xw) {
    const uint32_t o = ((uint32_t)min(xb, kb - 1) * 256u + (uint32_t)c16 * 16u) * 4u;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const u32x4 w4 = __builtin_amdgcn_raw_buffer_load_b128(xr, o + 16u * m, 0, 0);
      v[4 * m + 0] = __uint_as_float(w4.x);
      v[4 * m + 1] = __uint_as_float(w4.y);
      v[4 * m + 2] = __uint_as_float(w4.z);
      v[4 * m + 3] = __uint_as_float(w4.w);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  const MatRsrc mr[2] = {mat_rsrc(A.codes[0] + ec * A.stride_codes[0], A.scales[0] + ec * A.stride_scales[0], I, kb),
                         mat_rsrc(A.codes[1] + ec * A.stride_codes[1], A.scales[1] + ec * A.stride_scales[1], I, kb)};
  // loads in the order of use: every row's chunk of load 0, then of load 1, ...
  uint4 wr[2 * RPW][NL];  // [2r] gate row r, [2r + 1] up row r
#pragma unroll
  for (int i = 0; i < NL; ++i)
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const uint32_t srow = (uint32_t)min(row0 + r, I - 1) * (uint32_t)kb;
#pragma unroll
      for (int m = 0; m < 2; ++m)
        wr[2 * r + m][i] =
            buf_load16(mr[m].codes, (uint32_t)min(8 * i + g, kb - 1) * 128u + (uint32_t)cp * 16u, srow * 128u);
    }
  // after the block butterfly a lane keeps the row rev(lane bits): its scales
  uint16_t sr[2][NL];
  const int lrow = min(row0 + rev_bits<clog2(RPW)>(lane & (RPW - 1)), I - 1);
#pragma unroll
  for (int m = 0; m < 2; ++m) load_lane_scales<NL>(mr[m], lrow, kb, g, sr[m]);
  if (xw) quantize16_to_lds(v, min(xb, kb - 1), c16, s.q, s.d, s.b, xb < kb);
  for (int blk = xb + WAVES * 4; blk < kb; blk += WAVES * 4) {
    const uint32_t o = ((uint32_t)blk * 256u + (uint32_t)c16 * 16u) * 4u;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const u32x4 w4 = __builtin_amdgcn_raw_buffer_load_b128(xr, o + 16u * m, 0, 0);
      v[4 * m + 0] = __uint_as_float(w4.x);
      v[4 * m + 1] = __uint_as_float(w4.y);
      v[4 * m + 2] = __uint_as_float(w4.z);
      v[4 * m + 3] = __uint_as_float(w4.w);
    }
    quantize16_to_lds(v, blk, c16, s.q, s.d, s.b, true);
  }
  __syncthreads();
  if (stage) {  // stage buffers and the status word, once per call
    for (int i = threadIdx.x; i < kb * 64; i += WAVES * 64)
      reinterpret_cast<int*>(A.xq)[i] = reinterpret_cast<const int*>(s.q)[i];
    for (int i = threadIdx.x; i < kb; i += WAVES * 64) {
      A.xd[i] = s.d[i];
      A.xb[i] = s.b[i];
    }
    if (threadIdx.x == 0) {
      int bad = 0;
      for (int jj = 0; jj < A.topk; ++jj) bad |= (A.topk_idx[jj] < 0) | (A.topk_idx[jj] >= A.n_experts);
      A.ctrl[kFlags] = bad;
    }
  }
  if (!valid || row0 >= I) return;
  int qa[NL][8];
  lds_acts<NL>(s.q, kb, g, cp, qa);
  using RR = RowReduce<RPW, 2>;
  static_assert(RR::KI == 1, "a lane keeps one row after the block butterfly");
  float acc[2] = {0.0f, 0.0f};
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int b = 8 * i + g;
    const float dv = (!RAGGED || b < kb) ? s.d[min(b, kb - 1)] : 0.0f;
    int p[2 * RPW];
#pragma unroll
    for (int v = 0; v < 2 * RPW; ++v) p[v] = dot_chunk16(wr[v][i], qa[i]);
    RR::block_sums(p);
    // debug stage dump: the lane's kept row (one lane per row) stores the exact block sums
    if (A.dbg_gsum != nullptr && RR::block_writer(lane) && b < kb) {
      const int r = RR::kept(0, lane);
      if (row0 + r < I) {
        const int64_t o = ((int64_t)j * I + row0 + r) * kb + b;
        A.dbg_gsum[o] = p[0] >> 4;
        A.dbg_usum[o] = p[1] >> 4;
      }
    }
#pragma unroll
    for (int m = 0; m < 2; ++m) acc[m] = fmaf(f16_bits_to_f32(sr[m][i]) * dv, (float)(p[m] >> 4), acc[m]);
  }
  RR::block_totals(acc);
  const int r = RR::item(lane);
  if (RR::writer(lane) && row0 + r < I) {
    A.h[(int64_t)j * I + row0 + r] = silu_f32(acc[0]) * acc[1];
    if (A.dbg_g != nullptr) {
      A.dbg_g[(int64_t)j * I + row0 + r] = acc[0];
      A.dbg_u[(int64_t)j * I + row0 + r] = acc[1];
    }
  }
}

// Down of one single-token workgroup `wg`: one wave per slot (TOPK waves), wave j owning
// rows row0 .. row0 + ROWS - 1 of slot j's down matrix. A wave quantizes its own slot's h
// in registers (each 8-lane group holds one 256-block of it: the block's absmax and code
// sum come from group butterflies), so no wave waits for another before its dot products
// and each wave's arithmetic follows its own weight loads. Per load, the ROWS rows meet
// in the integer block butterfly; the lane that keeps a row applies the block's scales;
// the fp32 butterfly over blocks leaves one row per lane; the slots' row results meet in
// LDS, where ROWS lanes form out = sum_j w_j * y_j in ascending j.
// `stage`: this workgroup also stores the quantized h.
template <int NL, int ROWS, int TOPK, bool RAGGED>
__device__ __forceinline__ void t1_down_wg(const MoeArgs& A, float* __restrict__ out, int wg, bool stage,
                                           float* __restrict__ s_y) {
  static_assert(ROWS >= 1 && ROWS <= 32 && (ROWS & (ROWS - 1)) == 0, "rows per wave: a power of two <= 32");
  constexpr int NH = NL < 2 ? NL : 2;  // blocks of h loaded ahead of the weights
  const int lane = threadIdx.x & 63, j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 3, cp = lane & 7;
  const int kb = A.inter / 256, H = A.hidden, I = A.inter;
  const int row0 = wg * ROWS;
  const int e = A.topk_idx[j];
  using RR = RowReduce<ROWS, 1>;
  constexpr int KI = RR::KI;
  if (e >= 0 && e < A.n_experts && row0 < H) {  // wave-uniform: an unrouted slot's h is never written
    // the slot's h first (its waits must not queue behind the weights), then every weight load
    const __amdgpu_buffer_rsrc_t hr = make_rsrc(A.h + (int64_t)j * I, (uint32_t)I * 4u);
    float vh[NH][32];
#pragma unroll
    for (int i = 0; i < NH; ++i) buf_load32f(hr, (uint32_t)min(8 * i + g, kb - 1), cp, vh[i]);
    __builtin_amdgcn_sched_barrier(0);
    const MatRsrc mr = mat_rsrc(A.codes[2] + (int64_t)e * A.stride_codes[2], A.scales[2] + (int64_t)e * A.stride_scales[2],
                                H, kb);
    // loads in the order of use: every row's chunk of load 0, then of load 1, ...
    uint4 wr[ROWS][NL];
#pragma unroll
    for (int i = 0; i < NL; ++i)
#pragma unroll
      for (int r = 0; r < ROWS; ++r)
        wr[r][i] = buf_load16(mr.codes, (uint32_t)min(8 * i + g, kb - 1) * 128u + (uint32_t)cp * 16u,
                              (uint32_t)min(row0 + r, H - 1) * (uint32_t)kb * 128u);
    // after the block butterfly a lane keeps KI rows: their scales
    uint16_t sr[KI][NL];
#pragma unroll
    for (int k = 0; k < KI; ++k) {
      const uint32_t srow = (uint32_t)min(row0 + RR::kept(k, lane), H - 1) * (uint32_t)kb;
#pragma unroll
      for (int i = 0; i < NL; ++i) sr[k][i] = buf_load_u16(mr.scales, (srow + (uint32_t)min(8 * i + g, kb - 1)) * 2u, 0);
    }
    float acc[KI];
#pragma unroll
    for (int k = 0; k < KI; ++k) acc[k] = 0.0f;
#pragma unroll
    for (int i = 0; i < NL; ++i) {
      const int b = 8 * i + g;
      // block b of the slot's h: codes, scale and code sum (blocks past the row end repeat
      // the last block; their scale is taken as zero below and they are not stored)
      int qw[8], qs, bs;
      float dq;
      if (i < NH) {
        quantize_group32(vh[i < NH ? i : 0], qw, qs, dq, bs);
      } else {
        float v[32];
        buf_load32f(hr, (uint32_t)min(b, kb - 1), cp, v);
        quantize_group32(v, qw, qs, dq, bs);
      }
      if (stage && b < kb) {
        int4* qp = reinterpret_cast<int4*>(A.hq + (int64_t)j * I + b * 256 + cp * 32);
        qp[0] = make_int4(qw[0], qw[1], qw[2], qw[3]);
        qp[1] = make_int4(qw[4], qw[5], qw[6], qw[7]);
        if (cp == 0) {
          A.hd[j * kb + b] = dq;
          A.hb[j * kb + b] = bs;
        }
      }
      int p[ROWS];
#pragma unroll
      for (int r = 0; r < ROWS; ++r) p[r] = dot_chunk16(wr[r][i], qw);
      RR::block_sums(p);
      // debug stage dump: each kept row's exact block sum, one lane per (row, block)
      if (A.dbg_dsum != nullptr && RR::block_writer(lane) && b < kb) {
#pragma unroll
        for (int k = 0; k < KI; ++k) {
          const int r = RR::kept(k, lane);
          if (row0 + r < H) A.dbg_dsum[((int64_t)j * H + row0 + r) * kb + b] = p[k] >> 4;
        }
      }
      const float dv = (!RAGGED || b < kb) ? dq : 0.0f;
#pragma unroll
      for (int k = 0; k < KI; ++k) acc[k] = fmaf(f16_bits_to_f32(sr[k][i]) * dv, (float)(p[k] >> 4), acc[k]);
    }
    RR::block_totals(acc);
    if (RR::writer(lane)) s_y[j * ROWS + RR::item(lane)] = acc[0];
  }
  __syncthreads();
  const int t = threadIdx.x;
  if (t < ROWS && row0 + t < H) {
    float o = 0.0f;
#pragma unroll
    for (int jj = 0; jj < TOPK; ++jj) {
      const int ej = A.topk_idx[jj];
      if (ej < 0 || ej >= A.n_experts) continue;
      const float y = s_y[jj * ROWS + t];
      o = fmaf(A.topk_w[jj], y, o);
      A.yd[(int64_t)jj * H + row0 + t] = y;
    }
    out[row0 + t] = o;
  }
}

template <int NL, int RPW, int WAVES, bool RAGGED>
__global__ __launch_bounds__(WAVES * 64) void k_t1_gateup(const float* __restrict__ x, MoeArgs A) {
  __shared__ __attribute__((aligned(16))) uint8_t s_raw[kT1LdsBytes];
  t1_gateup_wg<NL, RPW, WAVES, RAGGED>(x, A, blockIdx.x, blockIdx.x == 0, T1Lds(s_raw));
}

template <int NL, int ROWS, int TOPK, bool RAGGED>
__global__ __launch_bounds__(TOPK * 64) void k_t1_down(MoeArgs A, float* __restrict__ out) {
  __shared__ float s_y[TOPK * ROWS];
  t1_down_wg<NL, ROWS, TOPK, RAGGED>(A, out, blockIdx.x, blockIdx.x == 0, s_y);
}

// ---------------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------------

using moe_fn = void (*)(MoeArgs);

constexpr int kMaxDevices = 64;  // per-device host state (side stream, compute units, scratch)

// Grouped-decode tiles: each wave holds about 16 unpacked chunks per lane
// (NMAT * RPW * NL), in kTbWaves-wave workgroups.
static int tb_rpw(int nmat, int nl) {
  if (nmat == 2) return nl == 1 ? 8 : (nl == 2 ? 4 : (nl <= 4 ? 2 : 1));
  return nl <= 2 ? 8 : (nl <= 4 ? 4 : 2);
}

#ifndef TQ_TB_NTL2
#define TQ_TB_NTL2 2
#endif
#ifndef TQ_TB_NTL4
#define TQ_TB_NTL4 1
#endif
// The grouped VALU kernel's tile for NL loads per lane: rows per wave (as tb_rpw), the
// first token group's width (pairs, single tokens where a pair's activations would crowd
// the registers that hold the weights) and the later groups' width.
template <int NMAT, int NL>
struct TbShape {
  static constexpr int RPW =
      NMAT == 2 ? (NL == 1 ? 8 : (NL == 2 ? 4 : (NL <= 4 ? 2 : 1))) : (NL <= 2 ? 8 : (NL <= 4 ? 4 : 2));
  static constexpr int NT = NL <= 2 ? 2 : 1;
  static constexpr int NTL = NL <= 2 ? TQ_TB_NTL2 : (NL <= 4 ? TQ_TB_NTL4 : 1);
};

template <int NMAT, int NL, bool R>
static moe_fn pick_tb_nl() {
  using S = TbShape<NMAT, NL>;
  return k_tb<NMAT, NL, S::RPW, S::NT, S::NTL, kTbWaves, R>;
}

template <int NMAT, bool R>
static moe_fn pick_tb_r(int nl) {
  switch (nl) {
    case 1: return pick_tb_nl<NMAT, 1, R>();
    case 2: return pick_tb_nl<NMAT, 2, R>();
    case 3: return pick_tb_nl<NMAT, 3, R>();
    case 4: return pick_tb_nl<NMAT, 4, R>();
    case 5: return pick_tb_nl<NMAT, 5, R>();
    case 6: return pick_tb_nl<NMAT, 6, R>();
    case 7: return pick_tb_nl<NMAT, 7, R>();
    default: return pick_tb_nl<NMAT, 8, R>();
  }
}

template <int NMAT>
static moe_fn pick_tb(int kb) {
  const int nl = (kb + 7) / 8;
  return kb % 8 == 0 ? pick_tb_r<NMAT, false>(nl) : pick_tb_r<NMAT, true>(nl);
}

// The mixed path's one-launch kernel: NL rounded up to 1, 2, 4 or 8 (the extra loads of
// a row reread its last block, whose scale is then taken as zero; the tile shapes of a
// rounded NL equal those of the exact one), which keeps the instances few.
using mixed_fn = void (*)(MoeArgs, int);
template <int NMAT, int NL>
static mixed_fn pick_mixed_nl(bool ragged) {
  using S = TbShape<NMAT, NL>;
  return ragged ? k_mixed<NMAT, NL, S::RPW, S::NT, S::NTL, true> : k_mixed<NMAT, NL, S::RPW, S::NT, S::NTL, false>;
}
template <int NMAT>
static mixed_fn pick_mixed(int kb) {
  const int nl = (kb + 7) / 8, nl4 = nl <= 2 ? nl : (nl <= 4 ? 4 : 8);
  const bool ragged = kb != 8 * nl4;
  switch (nl4) {
    case 1: return pick_mixed_nl<NMAT, 1>(ragged);
    case 2: return pick_mixed_nl<NMAT, 2>(ragged);
    case 4: return pick_mixed_nl<NMAT, 4>(ragged);
    default: return pick_mixed_nl<NMAT, 8>(ragged);
  }
}

// Compute units of the calling thread's current device (queried once per device).
static int device_cus() {
  static std::atomic<int> cache[kMaxDevices];
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 256;
  }
  int v = cache[dev].load(std::memory_order_relaxed);
  if (v == 0) {
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v < 8) {
      (void)hipGetLastError();
      v = 256;
    }
    cache[dev].store(v, std::memory_order_relaxed);
  }
  return v;
}

// Tile shapes of the single-token path (measured on MI355X; overridable at build time).
#ifndef TQ_T1_RPW_GU
#define TQ_T1_RPW_GU 4  // rows of gate and of up per wave
#endif
#ifndef TQ_T1_WAVES_GU
#define TQ_T1_WAVES_GU 4  // waves per gate/up workgroup
#endif
constexpr int kT1RpwGU = TQ_T1_RPW_GU;
constexpr int kT1WavesGU = TQ_T1_WAVES_GU;

using t1gu_fn = void (*)(const float*, MoeArgs);
using t1dn_fn = void (*)(MoeArgs, float*);

template <bool R>
static t1gu_fn pick_t1_gateup_r(int nl) {
  switch (nl) {
    case 1: return k_t1_gateup<1, kT1RpwGU, kT1WavesGU, R>;
    case 2: return k_t1_gateup<2, kT1RpwGU, kT1WavesGU, R>;
    case 3: return k_t1_gateup<3, (kT1RpwGU + 1) / 2, kT1WavesGU, R>;
    case 4: return k_t1_gateup<4, (kT1RpwGU + 1) / 2, kT1WavesGU, R>;
    case 5: return k_t1_gateup<5, 1, kT1WavesGU, R>;
    case 6: return k_t1_gateup<6, 1, kT1WavesGU, R>;
    case 7: return k_t1_gateup<7, 1, kT1WavesGU, R>;
    default: return k_t1_gateup<8, 1, kT1WavesGU, R>;
  }
}
// ragged: kb (blocks per row) not a multiple of 8, so the last 16-byte load of a row is
// partly past its end
static t1gu_fn pick_t1_gateup(int kb) {
  const int nl = (kb + 7) / 8;
  return kb % 8 ? pick_t1_gateup_r<true>(nl) : pick_t1_gateup_r<false>(nl);
}
static int t1_rpw_gu(int nl) { return nl <= 2 ? kT1RpwGU : (nl <= 4 ? (kT1RpwGU + 1) / 2 : 1); }

// Rows of down per wave (one wave per slot): 16 loads of 1 KB per wave at NL = 1 and
// eight or more slots, fewer rows with fewer slots (so that a step still has about 2048
// waves) or longer rows (so that a wave's chunks stay within its registers).
constexpr int t1_down_rows(int nl, int topk) {
  const int r = (16 / nl) * (topk < 4 ? topk : 4) / 4;
  return r < 1 ? 1 : 1 << clog2(r);  // rounded down to a power of two
}

template <int NL, bool R>
static t1dn_fn pick_t1_down_k(int topk) {
  switch (topk) {
    case 1: return k_t1_down<NL, t1_down_rows(NL, 1), 1, R>;
    case 2: return k_t1_down<NL, t1_down_rows(NL, 2), 2, R>;
    case 3: return k_t1_down<NL, t1_down_rows(NL, 3), 3, R>;
    case 4: return k_t1_down<NL, t1_down_rows(NL, 4), 4, R>;
    case 5: return k_t1_down<NL, t1_down_rows(NL, 5), 5, R>;
    case 6: return k_t1_down<NL, t1_down_rows(NL, 6), 6, R>;
    case 7: return k_t1_down<NL, t1_down_rows(NL, 7), 7, R>;
    default: return k_t1_down<NL, t1_down_rows(NL, 8), 8, R>;
  }
}

static int t1_down_nl(int kb) {
  const int nl = (kb + 7) / 8;
  return nl <= 2 ? nl : (nl <= 4 ? 4 : 8);
}

// topk * inter <= 16384 (the single-token path's bound) keeps NL <= 8.
template <bool R>
static t1dn_fn pick_t1_down_r(int nl, int topk) {
  switch (nl) {
    case 1: return pick_t1_down_k<1, R>(topk);
    case 2: return pick_t1_down_k<2, R>(topk);
    case 4: return pick_t1_down_k<4, R>(topk);
    default: return pick_t1_down_k<8, R>(topk);
  }
}
static t1dn_fn pick_t1_down(int kb, int topk) {
  const int nl = t1_down_nl(kb);
  // NL is rounded up to 4 or 8 for nl > 2: those loads may run past the row end too
  const bool ragged = kb % 8 != 0 || nl * 8 != kb;
  return ragged ? pick_t1_down_r<true>(nl, topk) : pick_t1_down_r<false>(nl, topk);
}

// One stage's kernel; with timing events, launched with hipExtLaunchKernelGGL so the
// start/stop events take the kernel's own dispatch timestamps.
template <typename F, typename... Args>
static tq_status launch_stage(void* const* events, int stage, F kernel, dim3 grid, int threads, hipStream_t st,
                              const char* fn, Args... args) {
  if (events)
    hipExtLaunchKernelGGL(kernel, grid, dim3(threads), 0, st, (hipEvent_t)events[2 * stage],
                          (hipEvent_t)events[2 * stage + 1], 0, args...);
  else
    hipLaunchKernelGGL(kernel, grid, dim3(threads), 0, st, args...);
  return check_launch(fn);
}

// A stage of two kernels on one stream (the start event before the first, the stop event
// after the second).
template <typename F1, typename F2, typename... Args>
static tq_status launch_stage2(void* const* events, int stage, F1 k1, dim3 g1, int t1, F2 k2, dim3 g2, int t2,
                               hipStream_t st, const char* fn, Args... args) {
  if (events) {
    hipExtLaunchKernelGGL(k1, g1, dim3(t1), 0, st, (hipEvent_t)events[2 * stage], nullptr, 0, args...);
    hipExtLaunchKernelGGL(k2, g2, dim3(t2), 0, st, nullptr, (hipEvent_t)events[2 * stage + 1], 0, args...);
  } else {
    hipLaunchKernelGGL(k1, g1, dim3(t1), 0, st, args...);
    hipLaunchKernelGGL(k2, g2, dim3(t2), 0, st, args...);
  }
  return check_launch(fn);
}

// A stage with no kernel of its own on this path: its event pair is recorded back to back.
static tq_status empty_stage(void* const* events, int stage, hipStream_t st, const char* fn) {
  if (!events) return TQ_OK;
  if (hipEventRecord((hipEvent_t)events[2 * stage], st) != hipSuccess ||
      hipEventRecord((hipEvent_t)events[2 * stage + 1], st) != hipSuccess)
    return fail(TQ_ERR_DEVICE, "%s: hipEventRecord failed", fn);
  return TQ_OK;
}

// The grouped MFMA path's second stream. Each projection runs as two launches that touch
// disjoint outputs (the 128-token tiles of the experts of more than kMTs slots, and the
// experts of at most kMTs slots): the first is bound by MFMA issue and LDS operand reads,
// the second by its weight stream, so the second runs beside the first on a stream the
// library owns (one per device, default priority), forked from the caller's stream and
// joined back to it by events (the mixed path's debug instances use it too; its
// production kernels run as one launch). It is created by the first such call on a
// device that is not being captured and may allocate (tq_moe_grouped_noalloc uses it
// only once it exists); until then, or if creating it failed, both launches run in order
// on the caller's stream. `mu` serializes the fork-launch-join sequences of callers on
// different host threads, which share the two events.
struct SideStream {
  std::mutex mu;
  bool tried = false;
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, join = nullptr;
};
static SideStream g_side[kMaxDevices];

static SideStream* side_stream(hipStream_t st, bool may_create) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return nullptr;
  }
  SideStream& ss = g_side[dev];
  std::lock_guard<std::mutex> lock(ss.mu);
  if (!ss.tried) {
    if (!may_create) return nullptr;
    hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
    if (hipStreamIsCapturing(st, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) {
      (void)hipGetLastError();
      return nullptr;  // (no stream or event is created inside a capture)
    }
    ss.tried = true;
    const bool ok = hipStreamCreateWithFlags(&ss.s, hipStreamNonBlocking) == hipSuccess &&
                    hipEventCreateWithFlags(&ss.fork, hipEventDisableTiming) == hipSuccess &&
                    hipEventCreateWithFlags(&ss.join, hipEventDisableTiming) == hipSuccess;
    if (!ok) {
      if (ss.join) (void)hipEventDestroy(ss.join);
      if (ss.fork) (void)hipEventDestroy(ss.fork);
      if (ss.s) (void)hipStreamDestroy(ss.s);
      ss.s = nullptr;
      ss.fork = ss.join = nullptr;
      (void)hipGetLastError();
    }
  }
  return ss.s ? &ss : nullptr;
}

// A stage of two independent kernels: k1 on `st`, k2 on the side stream, both after the
// work queued on `st` so far, with `st` waiting for both before anything queued after.
// With timing events the stage's pair is recorded on `st` before the fork and after the
// join (it spans both launches). Without a side stream: launch_stage2.
template <typename F1, typename F2, typename... Args>
static tq_status launch_pair(void* const* events, int stage, SideStream* ss, F1 k1, dim3 g1, int t1, F2 k2, dim3 g2,
                             int t2, hipStream_t st, const char* fn, Args... args) {
  if (!ss) return launch_stage2(events, stage, k1, g1, t1, k2, g2, t2, st, fn, args...);
  std::lock_guard<std::mutex> lock(ss->mu);
  if (events && hipEventRecord((hipEvent_t)events[2 * stage], st) != hipSuccess)
    return fail(TQ_ERR_DEVICE, "%s: hipEventRecord failed", fn);
  if (hipEventRecord(ss->fork, st) != hipSuccess || hipStreamWaitEvent(ss->s, ss->fork, 0) != hipSuccess)
    return fail(TQ_ERR_DEVICE, "%s: fork to the side stream failed", fn);
  hipLaunchKernelGGL(k1, g1, dim3(t1), 0, st, args...);
  hipLaunchKernelGGL(k2, g2, dim3(t2), 0, ss->s, args...);
  tq_status r = check_launch(fn);
  if (hipEventRecord(ss->join, ss->s) != hipSuccess || hipStreamWaitEvent(st, ss->join, 0) != hipSuccess)
    return fail(TQ_ERR_DEVICE, "%s: join from the side stream failed", fn);
  if (r != TQ_OK) return r;
  if (events && hipEventRecord((hipEvent_t)events[2 * stage + 1], st) != hipSuccess)
    return fail(TQ_ERR_DEVICE, "%s: hipEventRecord failed", fn);
  return TQ_OK;
}

static tq_status validate_experts(const tq_experts* ex, const char* fn) {
  if (!ex) return fail(TQ_ERR_INVALID, "%s: null experts descriptor", fn);
  if (ex->n_experts < 1 || ex->n_experts > kMaxExperts)
    return fail(TQ_ERR_INVALID, "%s: n_experts = %d outside [1, %d]", fn, ex->n_experts, kMaxExperts);
  for (int v : {ex->hidden, ex->inter})
    if (v <= 0 || v % 256 != 0 || v > kMaxK)
      return fail(TQ_ERR_INVALID, "%s: hidden = %d and inter = %d must be multiples of 256 in [256, %d]", fn, ex->hidden,
                  ex->inter, kMaxK);
  const uint8_t* cs[3] = {ex->gate_codes, ex->up_codes, ex->down_codes};
  const uint16_t* ss[3] = {ex->gate_scales, ex->up_scales, ex->down_scales};
  for (int p = 0; p < 3; ++p) {
    if (!cs[p] || !ss[p]) return fail(TQ_ERR_INVALID, "%s: null expert codes or scales", fn);
    if (!aligned(cs[p], 128) || ex->stride_codes[p] % 128 != 0)
      return fail(TQ_ERR_ALIGN, "%s: expert codes pointers and byte strides must be multiples of 128", fn);
    if (!aligned(ss[p], 2)) return fail(TQ_ERR_ALIGN, "%s: expert scales must be 2-byte aligned", fn);
    if (ex->n_experts > 1 && (ex->stride_codes[p] <= 0 || ex->stride_scales[p] <= 0))
      return fail(TQ_ERR_INVALID, "%s: expert strides must be positive", fn);
  }
  return TQ_OK;
}

// The path a call takes (see tq_moe_path in tq.h).
static int choose_path(const tq_experts* ex, int64_t t, int32_t topk, int32_t flags) {
  if (t == 1 && topk <= kT1MaxTopk && (int64_t)topk * ex->inter <= kT1MaxHq && !(flags & TQ_MOE_FORCE_MFMA))
    return TQ_MOE_PATH_T1;
  // (both grouped paths address the quantized activations with 32-bit buffer offsets)
  const int64_t S = t * topk;
  if (S * std::max(ex->hidden, ex->inter) >= ((int64_t)1 << 31)) return -1;
  if ((flags & TQ_MOE_FORCE_MFMA) || (!(flags & TQ_MOE_FORCE_VALU) && S >= kMfmaMinSlots)) return TQ_MOE_PATH_MFMA;
  // (with at most kHybMin tokens no expert has more slots, duplicated ids aside)
  return !(flags & TQ_MOE_FORCE_VALU) && t > kHybMin ? TQ_MOE_PATH_MIXED : TQ_MOE_PATH_VALU;
}

static tq_status moe_run(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                         const float* topk_w, int32_t topk, float* out, void* ws, size_t ws_bytes, int32_t flags,
                         void* stream, void* const* events, const char* fn, bool may_allocate = true) {
  clear_error();
  tq_status st = validate_experts(ex, fn);
  if (st != TQ_OK) return st;
  if (t < 0 || t > (1 << 20)) return fail(TQ_ERR_INVALID, "%s: t = %lld outside [0, 2^20]", fn, (long long)t);
  if (topk < 1 || topk > kMaxTopk || topk > ex->n_experts)
    return fail(TQ_ERR_INVALID, "%s: topk = %d outside [1, min(%d, n_experts)]", fn, topk, kMaxTopk);
  if (flags & ~(TQ_MOE_FORCE_VALU | TQ_MOE_FORCE_MFMA | TQ_MOE_DEBUG_STAGES) ||
      (flags & (TQ_MOE_FORCE_VALU | TQ_MOE_FORCE_MFMA)) == (TQ_MOE_FORCE_VALU | TQ_MOE_FORCE_MFMA))
    return fail(TQ_ERR_INVALID, "%s: bad flags 0x%x", fn, flags);
  const bool debug = (flags & TQ_MOE_DEBUG_STAGES) != 0;
  if (t == 0) {
    for (int i = 0; i < kNumStages; ++i)
      if ((st = empty_stage(events, i, (hipStream_t)stream, fn)) != TQ_OK) return st;
    return TQ_OK;
  }
  if (!x || !topk_idx || !topk_w || !out || !ws) return fail(TQ_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(x, 16) || !aligned(out, 16) || !aligned(ws, 256) || !aligned(topk_idx, 4) || !aligned(topk_w, 4))
    return fail(TQ_ERR_ALIGN, "%s: x and out must be 16-byte aligned, ws 256-byte aligned", fn);
  const Layout L = make_layout(ex->n_experts, ex->hidden, ex->inter, t, topk);
  const size_t need = debug ? L.total_dbg : L.total;
  if (ws_bytes < need)
    return fail(TQ_ERR_WORKSPACE, "%s: workspace %zu bytes < required %zu%s", fn, ws_bytes, need,
                debug ? " (with the debug stage dump)" : "");

  uint8_t* base = static_cast<uint8_t*>(ws);
  MoeArgs A{};
  A.n_experts = ex->n_experts;
  A.hidden = ex->hidden;
  A.inter = ex->inter;
  A.topk = topk;
  A.t = t;
  A.codes[0] = ex->gate_codes;
  A.codes[1] = ex->up_codes;
  A.codes[2] = ex->down_codes;
  A.scales[0] = ex->gate_scales;
  A.scales[1] = ex->up_scales;
  A.scales[2] = ex->down_scales;
  for (int p = 0; p < 3; ++p) {
    A.stride_codes[p] = ex->stride_codes[p];
    A.stride_scales[p] = ex->stride_scales[p];
  }
  A.topk_idx = topk_idx;
  A.topk_w = topk_w;
  A.ctrl = reinterpret_cast<int32_t*>(base + L.ctrl);
  A.active = reinterpret_cast<int32_t*>(base + L.active);
  A.act_off = reinterpret_cast<int32_t*>(base + L.act_off);
  A.tt_off = reinterpret_cast<int32_t*>(base + L.tt_off);
  A.tile_exp = reinterpret_cast<int32_t*>(base + L.tile_exp);
  A.tt32_off = reinterpret_cast<int32_t*>(base + L.tt32_off);
  A.tile32_exp = reinterpret_cast<int32_t*>(base + L.tile32_exp);
  A.slot_list = reinterpret_cast<int32_t*>(base + L.slot_list);
  A.xq = reinterpret_cast<int8_t*>(base + L.xq);
  A.xd = reinterpret_cast<float*>(base + L.xd);
  A.xb = reinterpret_cast<int32_t*>(base + L.xb);
  A.h = reinterpret_cast<float*>(base + L.h);
  A.hq = reinterpret_cast<int8_t*>(base + L.hq);
  A.hd = reinterpret_cast<float*>(base + L.hd);
  A.hb = reinterpret_cast<int32_t*>(base + L.hb);
  A.yd = reinterpret_cast<float*>(base + L.yd);
  if (debug) {
    A.dbg_g = reinterpret_cast<float*>(base + L.dg);
    A.dbg_u = reinterpret_cast<float*>(base + L.du);
    A.dbg_gsum = reinterpret_cast<int32_t*>(base + L.dgs);
    A.dbg_usum = reinterpret_cast<int32_t*>(base + L.dus);
    A.dbg_dsum = reinterpret_cast<int32_t*>(base + L.dds);
  }

  const int nl_gu = (ex->hidden / 256 + 7) / 8, nl_dn = (ex->inter / 256 + 7) / 8;
  const int tr_gu = kTbWaves * tb_rpw(2, nl_gu), tr_dn = kTbWaves * tb_rpw(1, nl_dn);
  A.tiles_gu = (ex->inter + tr_gu - 1) / tr_gu;
  A.tiles_dn = (ex->hidden + tr_dn - 1) / tr_dn;
  const int64_t S = t * topk;
  const int64_t max_active = std::min<int64_t>(S, ex->n_experts);
  const int64_t cap = 256 * 16;  // workgroups per launch; the rest are strided over them
  const unsigned g_gu = (unsigned)std::min<int64_t>(max_active * A.tiles_gu, cap);
  const unsigned g_dn = (unsigned)std::min<int64_t>(max_active * A.tiles_dn, cap);
  const int64_t xblocks = t * (ex->hidden / 256), hblocks = S * (ex->inter / 256);
  const int nq = (int)((xblocks + 31) / 32);
  hipStream_t stm = (hipStream_t)stream;

  (void)hipGetLastError();
  const int path = choose_path(ex, t, topk, flags);
  if (path < 0)
    return fail(TQ_ERR_INVALID, "%s: t * topk * max(hidden, inter) = %lld * %d reaches 2^31 (32-bit activation offsets)",
                fn, (long long)S, std::max(ex->hidden, ex->inter));
  if (path == TQ_MOE_PATH_T1) {
    const int rgu = t1_rpw_gu(nl_gu);
    // single token: gate_up, then down with the requant and the combine fused; the
    // prologue, requant and combine stages are empty on this path
    A.tiles_gu = (ex->inter + kT1WavesGU * rgu - 1) / (kT1WavesGU * rgu);
    const int rows_dn = t1_down_rows(t1_down_nl(ex->inter / 256), topk);
    const unsigned tiles_dn = (unsigned)((ex->hidden + rows_dn - 1) / rows_dn);
    if ((st = empty_stage(events, 0, stm, fn)) != TQ_OK) return st;
    if ((st = launch_stage(events, 1, pick_t1_gateup(ex->hidden / 256), dim3((unsigned)(topk * A.tiles_gu)), kT1WavesGU * 64, stm,
                           fn, x, A)) != TQ_OK)
      return st;
    if ((st = empty_stage(events, 2, stm, fn)) != TQ_OK) return st;
    if ((st = launch_stage(events, 3, pick_t1_down(ex->inter / 256, topk), dim3(tiles_dn), topk * 64, stm, fn, A, out)) !=
        TQ_OK)
      return st;
    return empty_stage(events, 4, stm, fn);
  }
  // per-expert contraction on MFMA for prefill-sized groups (or when forced), VALU dot4
  // otherwise
  const bool mfma = path == TQ_MOE_PATH_MFMA, mixed = path == TQ_MOE_PATH_MIXED;
  A.hyb = mixed ? kHybMin : 0;
  A.tiles_mgu = (ex->inter + kMN - 1) / kMN;
  A.tiles_mdn = (ex->hidden + 2 * kMN - 1) / (2 * kMN);  // (two 16-row tiles per wave)
  A.tiles_mgus = (ex->inter + kMNs - 1) / kMNs;
  A.tiles_mdns = (ex->hidden + 2 * kMNs - 1) / (2 * kMNs);
  const int64_t max_tiles = S / kMT + max_active;
#ifndef TQ_MFMA_GRID
#define TQ_MFMA_GRID (256 * 16)
#endif
  // Beside the small-tile launch, the 128-token launch keeps five eighths of the compute
  // units (a multiple of 8 workgroups, one per unit, striding over the tasks); the other
  // units run the small tiles, and so do the first ones as they free up.
  // (the mixed path runs one launch per projection; only its debug instances, kept out
  // of that launch, take the side stream)
  SideStream* ss = mfma || (mixed && debug) ? side_stream(stm, may_allocate) : nullptr;
  const int64_t big_cap = ss ? std::max(8, device_cus() * 5 / 8 / 8 * 8) : TQ_MFMA_GRID;
  const unsigned g_mgu = (unsigned)std::min<int64_t>(max_tiles * A.tiles_mgu, big_cap);
  const unsigned g_mdn = (unsigned)std::min<int64_t>(max_tiles * A.tiles_mdn, big_cap);
  // (one tile per expert of at most kMTs slots)
  const unsigned g_mgus = (unsigned)std::min<int64_t>(max_active * A.tiles_mgus, TQ_MFMA_GRID);
  const unsigned g_mdns = (unsigned)std::min<int64_t>(max_active * A.tiles_mdns, TQ_MFMA_GRID);
  // mixed path, one launch: at most one MFMA-role workgroup per compute unit (a multiple
  // of 8, striding over the tasks; they come first, so the longest tasks start first)
  const int cus8 = std::max(8, device_cus() / 8 * 8);
  const int n_mgus = (int)std::min<int64_t>((max_active * A.tiles_mgus + 7) / 8 * 8, cus8);
  const int n_mdns = (int)std::min<int64_t>((max_active * A.tiles_mdns + 7) / 8 * 8, cus8);
  if ((st = launch_stage(events, 0, k_moe_prologue, dim3(nq + 1), 256, stm, fn, x, A)) != TQ_OK) return st;
  if (mfma && debug)
    st = launch_pair(events, 1, ss, k_moe_mfma<2, kMT, kMWaves, false, true>, dim3(g_mgu), kMWaves * 64,
                       k_moe_mfma<2, kMTs, kMWavesS, true, true>, dim3(g_mgus), kMWavesS * 64, stm, fn, A);
  else if (mfma)
    st = launch_pair(events, 1, ss, k_moe_mfma<2, kMT, kMWaves, false, false>, dim3(g_mgu), kMWaves * 64,
                       k_moe_mfma<2, kMTs, kMWavesS, true, false>, dim3(g_mgus), kMWavesS * 64, stm, fn, A);
  else if (mixed && !debug)
    st = launch_stage(events, 1, pick_mixed<2>(ex->hidden / 256), dim3((unsigned)n_mgus + g_gu), kTbWaves * 64, stm, fn,
                      A, n_mgus);
  else if (mixed)  // (debug: the VALU kernel on the caller's stream, the MFMA tiles beside it)
    st = launch_pair(events, 1, ss, pick_tb<2>(ex->hidden / 256), dim3(g_gu), kTbWaves * 64,
                     k_moe_mfma<2, kMTs, kMWavesS, true, true, false, true>, dim3(g_mgus), kMWavesS * 64, stm, fn, A);
  else st = launch_stage(events, 1, pick_tb<2>(ex->hidden / 256), dim3(g_gu), kTbWaves * 64, stm, fn, A);
  if (st != TQ_OK) return st;
  if ((st = launch_stage(events, 2, k_moe_requant, dim3((unsigned)((hblocks + 31) / 32)), 256, stm, fn, A, hblocks)) !=
      TQ_OK)
    return st;
  if (mfma && debug)
    st = launch_pair(events, 3, ss, k_moe_mfma<2, kMT, kMWaves, false, true, true>, dim3(g_mdn), kMWaves * 64,
                       k_moe_mfma<2, kMTs, kMWavesS, true, true, true>, dim3(g_mdns), kMWavesS * 64, stm, fn, A);
  else if (mfma)
    st = launch_pair(events, 3, ss, k_moe_mfma<2, kMT, kMWaves, false, false, true>, dim3(g_mdn), kMWaves * 64,
                       k_moe_mfma<2, kMTs, kMWavesS, true, false, true>, dim3(g_mdns), kMWavesS * 64, stm, fn, A);
  else if (mixed && !debug)
    st = launch_stage(events, 3, pick_mixed<1>(ex->inter / 256), dim3((unsigned)n_mdns + g_dn), kTbWaves * 64, stm, fn,
                      A, n_mdns);
  else if (mixed)
    st = launch_pair(events, 3, ss, pick_tb<1>(ex->inter / 256), dim3(g_dn), kTbWaves * 64,
                     k_moe_mfma<2, kMTs, kMWavesS, true, true, true, true>, dim3(g_mdns), kMWavesS * 64, stm, fn, A);
  else st = launch_stage(events, 3, pick_tb<1>(ex->inter / 256), dim3(g_dn), kTbWaves * 64, stm, fn, A);
  if (st != TQ_OK) return st;
  const int64_t nout = t * (ex->hidden / 4);
  if ((st = launch_stage(events, 4, k_moe_combine, dim3((unsigned)((nout + 255) / 256)), 256, stm, fn, A, out)) != TQ_OK)
    return st;
  return TQ_OK;
}

}  // namespace tq

extern "C" size_t tq_moe_workspace_bytes(const tq_experts* ex, int64_t t, int32_t topk) {
  if (!ex || ex->n_experts < 1 || ex->hidden <= 0 || ex->inter <= 0 || t < 0 || topk < 1) return 0;
  return tq::make_layout(ex->n_experts, ex->hidden, ex->inter, t, topk).total;
}

extern "C" tq_status tq_moe_workspace_layout(const tq_experts* ex, int64_t t, int32_t topk, tq_moe_layout* out) {
  using namespace tq;
  clear_error();
  tq_status st = validate_experts(ex, "tq_moe_workspace_layout");
  if (st != TQ_OK) return st;
  if (!out || t < 0 || topk < 1) return fail(TQ_ERR_INVALID, "tq_moe_workspace_layout: bad arguments");
  const Layout L = make_layout(ex->n_experts, ex->hidden, ex->inter, t, topk);
  out->xq = L.xq;
  out->xd = L.xd;
  out->xb = L.xb;
  out->h = L.h;
  out->hq = L.hq;
  out->hd = L.hd;
  out->hb = L.hb;
  out->yd = L.yd;
  out->flags = L.ctrl + 4 * kFlags;
  out->total = L.total;
  out->n_active = L.ctrl + 4 * kNActive;
  out->active = L.active;
  out->act_off = L.act_off;
  out->slot_list = L.slot_list;
  out->g = L.dg;
  out->u = L.du;
  out->gsum = L.dgs;
  out->usum = L.dus;
  out->dsum = L.dds;
  out->total_debug = L.total_dbg;
  return TQ_OK;
}

extern "C" tq_status tq_moe_grouped(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                                    const float* topk_w, int32_t topk, float* out, void* ws, size_t ws_bytes,
                                    int32_t flags, void* stream) {
  return tq::moe_run(ex, x, t, topk_idx, topk_w, topk, out, ws, ws_bytes, flags, stream, nullptr, "tq_moe_grouped");
}

// ---------------------------------------------------------------------------------
// A variant of tq_moe_grouped that allocates nothing: its workspace is a fixed device
// array, one per GPU, that lives until the process ends. Host code never passes the
// array's name to a kernel (on the host it only stands for the symbol): the device
// address comes from hipGetSymbolAddress, once per device, with that device current.
// ---------------------------------------------------------------------------------
namespace tq {

constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;

static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

// The calling thread's current device's copy of `scratch` (looked up on the first call on
// that device).
static tq_status scratch_ptr(void** out, const char* fn) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(TQ_ERR_DEVICE, "%s: hipGetDevice failed: %s", fn, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(TQ_ERR_DEVICE, "%s: device %d beyond %d", fn, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(TQ_ERR_DEVICE, "%s: hipGetSymbolAddress(scratch) failed on device %d: %s", fn, dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return TQ_OK;
}

}  // namespace tq

extern "C" size_t tq_moe_noalloc_max_bytes(void) { return tq::kNoAllocScratchBytes; }

extern "C" tq_status tq_moe_grouped_noalloc(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                                            const float* topk_w, int32_t topk, float* out, int32_t flags,
                                            void* stream) {
  using namespace tq;
  const char* fn = "tq_moe_grouped_noalloc";
  clear_error();
  tq_status st = validate_experts(ex, fn);
  if (st != TQ_OK) return st;
  if (t < 0 || topk < 1) return fail(TQ_ERR_INVALID, "%s: bad t = %lld or topk = %d", fn, (long long)t, topk);
  const Layout L = make_layout(ex->n_experts, ex->hidden, ex->inter, t, topk);
  const size_t need = (flags & TQ_MOE_DEBUG_STAGES) ? L.total_dbg : L.total;
  if (need > kNoAllocScratchBytes)
    return fail(TQ_ERR_WORKSPACE,
                "%s: this call needs %zu bytes of scratch, more than the fixed %zu (fewer tokens per call, or "
                "tq_moe_grouped with a caller workspace)",
                fn, need, kNoAllocScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_ptr(&ws, fn)) != TQ_OK) return st;
  return moe_run(ex, x, t, topk_idx, topk_w, topk, out, ws, kNoAllocScratchBytes, flags, stream, nullptr, fn,
                 /*may_allocate=*/false);
}

extern "C" int32_t tq_moe_path(const tq_experts* ex, int64_t t, int32_t topk, int32_t flags) {
  using namespace tq;
  clear_error();
  if (validate_experts(ex, "tq_moe_path") != TQ_OK) return -1;
  if (t < 1 || topk < 1 || topk > kMaxTopk || topk > ex->n_experts) {
    fail(TQ_ERR_INVALID, "tq_moe_path: bad t or topk");
    return -1;
  }
  return choose_path(ex, t, topk, flags);
}

extern "C" int32_t tq_moe_stage_count(void) { return tq::kNumStages; }

extern "C" const char* tq_moe_stage_name(int32_t i) {
  return (i >= 0 && i < tq::kNumStages) ? tq::kStageNames[i] : "";
}

extern "C" tq_status tq_moe_grouped_timed(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                                          const float* topk_w, int32_t topk, float* out, void* ws, size_t ws_bytes,
                                          int32_t flags, void* stream, void* const* events) {
  if (!events) return tq::fail(TQ_ERR_INVALID, "tq_moe_grouped_timed: events may not be NULL");
  for (int i = 0; i < 2 * tq::kNumStages; ++i)
    if (!events[i]) return tq::fail(TQ_ERR_INVALID, "tq_moe_grouped_timed: null event %d", i);
  return tq::moe_run(ex, x, t, topk_idx, topk_w, topk, out, ws, ws_bytes, flags, stream, events,
                     "tq_moe_grouped_timed");
}

extern "C" tq_status tq_moe_status(const void* ws, const tq_experts* ex, int64_t t, int32_t topk, int32_t* flags_out,
                                   void* stream) {
  using namespace tq;
  clear_error();
  if (!ws || !flags_out) return fail(TQ_ERR_INVALID, "tq_moe_status: null pointer");
  tq_status st = validate_experts(ex, "tq_moe_status");
  if (st != TQ_OK) return st;
  const Layout L = make_layout(ex->n_experts, ex->hidden, ex->inter, t, topk);
  hipError_t e = hipStreamSynchronize((hipStream_t)stream);
  if (e != hipSuccess) return fail(TQ_ERR_DEVICE, "tq_moe_status: stream error: %s", hipGetErrorString(e));
  int32_t ctrl[kCtrlWords];
  e = hipMemcpy(ctrl, static_cast<const uint8_t*>(ws) + L.ctrl, sizeof(ctrl), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(TQ_ERR_DEVICE, "tq_moe_status: copy failed: %s", hipGetErrorString(e));
  *flags_out = ctrl[kFlags];
  return TQ_OK;
}
