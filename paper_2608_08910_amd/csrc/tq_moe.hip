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

#include "tq_device.hpp"
#include "tq_internal.hpp"

namespace tq {

constexpr int kMaxExperts = 4096;
constexpr int kMaxTopk = 64;
constexpr int kNumStages = 5;
static const char* const kStageNames[kNumStages] = {"prologue", "gate_up", "requant", "down", "combine"};

// Control words at the start of the workspace.
enum Ctrl { kFlags = 0, kNActive = 1, kTasksGU = 2, kTasksDn = 3, kNValid = 4, kTasksMGU = 5, kTasksMDn = 6, kCtrlWords = 64 };

constexpr int kMT = 64;  // tokens per MFMA tile (four 16-row MFMA tiles)
constexpr int kMN = 64;  // weight rows per MFMA workgroup (four waves x 16)
constexpr int64_t kMfmaMinSlots = 1024;  // automatic path choice: MFMA from this many slots

struct Layout {
  size_t ctrl, active, act_off, tt_off, slot_list, xq, xd, xb, h, hq, hd, hb, yd, total;
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

// Loads are issued unconditionally from clamped (always valid) addresses and invalid
// lanes are zeroed with a select afterwards: a predicated load becomes a branch, and the
// compiler then waits for each load before issuing the next.

// The lane's activation slice of one token: for load i, block 8i + g, chunk cp. The row
// pointers are those of a valid token; `ok` zeroes the slice.
template <int NL>
__device__ __forceinline__ void load_acts(const int8_t* __restrict__ qrow, const float* __restrict__ drow,
                                          const int32_t* __restrict__ brow, int kb, int g, int cp, bool ok,
                                          int (&qa)[NL][8], float (&dd)[NL], int (&bb)[NL]) {
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int b = 8 * i + g;
    const bool v = ok && b < kb;
    const int bc = b < kb ? b : kb - 1;
    const int4* p = reinterpret_cast<const int4*>(qrow + bc * 256 + cp * 32);
    const int4 lo = p[0], hi = p[1];
    const float dv = drow[bc];
    const int bv = brow[bc];
    qa[i][0] = v ? lo.x : 0; qa[i][1] = v ? lo.y : 0; qa[i][2] = v ? lo.z : 0; qa[i][3] = v ? lo.w : 0;
    qa[i][4] = v ? hi.x : 0; qa[i][5] = v ? hi.y : 0; qa[i][6] = v ? hi.z : 0; qa[i][7] = v ? hi.w : 0;
    dd[i] = v ? dv : 0.0f;
    bb[i] = v ? bv : 0;
  }
}

// One row's lane slice of codes and scales; rowcodes/rowscales point at a valid row.
template <int NL>
__device__ __forceinline__ void load_row(const uint8_t* __restrict__ rowcodes, const uint16_t* __restrict__ rowscales,
                                         int kb, int g, int cp, bool ok, uint4 (&w)[NL], float (&s)[NL]) {
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int b = 8 * i + g;
    const bool v = ok && b < kb;
    const int bc = b < kb ? b : kb - 1;
    const uint4 raw = ldg16(rowcodes + bc * 128 + cp * 16);
    const float sv = f16_bits_to_f32(rowscales[bc]);
    w[i] = v ? raw : make_uint4(0, 0, 0, 0);
    s[i] = v ? sv : 0.0f;
  }
}

// One row against one token: exact block sums, one multiply-add per block, wave total.
template <int NL>
__device__ __forceinline__ float row_dot(const uint4 (&w)[NL], const float (&s)[NL], const int (&qa)[NL][8],
                                         const float (&dd)[NL], const int (&bb)[NL]) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int is = group_sum_i32(dot_chunk_u(w[i], qa[i])) - 4 * bb[i];
    acc = fmaf(s[i] * dd[i], (float)is, acc);
  }
  return wave_sum_groups_f32(acc);
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
  int32_t* slot_list;
  int8_t* xq;
  float* xd;
  int32_t* xb;
  float* h;
  int8_t* hq;
  float* hd;
  int32_t* hb;
  float* yd;
  int tiles_gu, tiles_dn;    // row tiles of the VALU kernels
  int tiles_mgu, tiles_mdn;  // row tiles of the MFMA kernels
};

// ---------------------------------------------------------------------------------
// prologue: quantize x (workgroups 0 .. nq-1) + dispatch (last workgroup)
// ---------------------------------------------------------------------------------

__global__ __launch_bounds__(256) void k_moe_prologue(const float* __restrict__ x, MoeArgs A, int nq) {
  if ((int)blockIdx.x < nq) {
    const int64_t nblocks = A.t * (A.hidden / 256);
    quantize_wave_blocks(x, nblocks, (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6), A.xq, A.xd, A.xb);
    return;
  }
  __shared__ int s_cnt[kMaxExperts];   // slots per expert
  __shared__ int s_base[kMaxExperts];  // rank of an active expert, then its slot cursor
  __shared__ int s_ebr[kMaxExperts];   // expert of each rank
  __shared__ int s_scan[256], s_scan2[256];
  __shared__ int s_nact, s_bad;
  const int tid = threadIdx.x, E = A.n_experts;
  const int64_t S = A.t * A.topk;
  for (int e = tid; e < E; e += 256) s_cnt[e] = 0;
  if (tid == 0) {
    s_bad = 0;
    s_nact = 0;
  }
  __syncthreads();
  for (int64_t s = tid; s < S; s += 256) {
    const int e = A.topk_idx[s];
    if (e >= 0 && e < E) atomicAdd(&s_cnt[e], 1);
    else s_bad = 1;
  }
  __syncthreads();
  // Rank the active experts. With more than one token per step, hottest first (count
  // descending, id ascending): the work queues below hand out tasks in rank order, so
  // the longest tasks start first, one per workgroup. One token: id order.
  const bool by_count = A.t > 1 && E <= 1024;
  for (int e = tid; e < E; e += 256) {
    const int c = s_cnt[e];
    int r = -1;
    if (c > 0) {
      r = 0;
      if (by_count) {
        for (int e2 = 0; e2 < E; ++e2) {
          const int c2 = s_cnt[e2];
          r += (c2 > c) | ((c2 == c) & (e2 < e));
        }
      } else {
        for (int e2 = 0; e2 < e; ++e2) r += s_cnt[e2] > 0;
      }
      s_ebr[r] = e;
      atomicAdd(&s_nact, 1);
    }
    s_base[e] = r;
  }
  __syncthreads();
  const int n_active = s_nact;
  // exclusive scan of the slot counts in rank order, contiguous ranks per thread
  const int per = (n_active + 255) / 256;
  const int r0 = min(n_active, tid * per), r1 = min(n_active, r0 + per);
  // (and of the kMT-token tiles of the MFMA path)
  int ns = 0, nt = 0;
  for (int r = r0; r < r1; ++r) {
    ns += s_cnt[s_ebr[r]];
    nt += (s_cnt[s_ebr[r]] + kMT - 1) / kMT;
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
    A.active[r] = e;
    A.act_off[r] = pos;
    A.tt_off[r] = tpos;
    s_base[e] = pos;  // rank no longer needed: becomes the expert's slot cursor
    pos += s_cnt[e];
    tpos += (s_cnt[e] + kMT - 1) / kMT;
  }
  if (tid == 255) {
    const int n_valid = s_scan[255], n_tiles = s_scan2[255];
    A.act_off[n_active] = n_valid;
    A.tt_off[n_active] = n_tiles;
    A.ctrl[kNActive] = n_active;
    A.ctrl[kNValid] = n_valid;
    A.ctrl[kTasksGU] = n_active * A.tiles_gu;
    A.ctrl[kTasksDn] = n_active * A.tiles_dn;
    A.ctrl[kTasksMGU] = n_tiles * A.tiles_mgu;
    A.ctrl[kTasksMDn] = n_tiles * A.tiles_mdn;
    A.ctrl[kFlags] = s_bad ? 1 : 0;
  }
  __syncthreads();
  for (int64_t s = tid; s < S; s += 256) {
    const int e = A.topk_idx[s];
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

// ---------------------------------------------------------------------------------
// gate_up: h[slot][row] = SiLU(Wg[e] xq) * (Wu[e] xq)
// ---------------------------------------------------------------------------------

template <int NL, int NT, int RPW>
__global__ __launch_bounds__(256) void k_moe_gateup(MoeArgs A) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int g = lane >> 3, cp = lane & 7;
  const int kb = A.hidden / 256, I = A.inter;
  const int n_tasks = A.ctrl[kTasksGU];
  for (int task = blockIdx.x; task < n_tasks; task += gridDim.x) {
    const int a = task / A.tiles_gu, tile = task - a * A.tiles_gu;
    const int64_t e = A.active[a];
    const int off = A.act_off[a], cnt = A.act_off[a + 1] - off;
    const int row0 = (tile * 4 + wv) * RPW;
    if (row0 >= I) continue;
    const uint8_t* gc = A.codes[0] + e * A.stride_codes[0];
    const uint8_t* uc = A.codes[1] + e * A.stride_codes[1];
    const uint16_t* gs = A.scales[0] + e * A.stride_scales[0];
    const uint16_t* us = A.scales[1] + e * A.stride_scales[1];
    uint4 wg[RPW][NL], wu[RPW][NL];
    float sg[RPW][NL], su[RPW][NL];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int64_t row = min(row0 + r, I - 1);
      load_row<NL>(gc + row * kb * 128, gs + row * kb, kb, g, cp, row0 + r < I, wg[r], sg[r]);
      load_row<NL>(uc + row * kb * 128, us + row * kb, kb, g, cp, row0 + r < I, wu[r], su[r]);
    }
    for (int c0 = 0; c0 < cnt; c0 += NT) {
      int qa[NT][NL][8];
      float dd[NT][NL];
      int bb[NT][NL];
      int slot[NT];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const bool ok = c0 + tt < cnt;
        slot[tt] = A.slot_list[off + min(c0 + tt, cnt - 1)];
        const int64_t tok = slot[tt] / A.topk;
        load_acts<NL>(A.xq + tok * A.hidden, A.xd + tok * kb, A.xb + tok * kb, kb, g, cp, ok, qa[tt], dd[tt], bb[tt]);
      }
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          const float gv = row_dot<NL>(wg[r], sg[r], qa[tt], dd[tt], bb[tt]);
          const float uv = row_dot<NL>(wu[r], su[r], qa[tt], dd[tt], bb[tt]);
          if (lane == 0 && c0 + tt < cnt && row0 + r < I) A.h[(int64_t)slot[tt] * I + row0 + r] = silu_f32(gv) * uv;
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------------
// down: yd[slot][row] = Wd[e] hq[slot]
// ---------------------------------------------------------------------------------

template <int NL, int NT, int RPW>
__global__ __launch_bounds__(256) void k_moe_down(MoeArgs A) {
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int g = lane >> 3, cp = lane & 7;
  const int kb = A.inter / 256, H = A.hidden;
  const int n_tasks = A.ctrl[kTasksDn];
  for (int task = blockIdx.x; task < n_tasks; task += gridDim.x) {
    const int a = task / A.tiles_dn, tile = task - a * A.tiles_dn;
    const int64_t e = A.active[a];
    const int off = A.act_off[a], cnt = A.act_off[a + 1] - off;
    const int row0 = (tile * 4 + wv) * RPW;
    if (row0 >= H) continue;
    const uint8_t* dc = A.codes[2] + e * A.stride_codes[2];
    const uint16_t* ds = A.scales[2] + e * A.stride_scales[2];
    uint4 w[RPW][NL];
    float s[RPW][NL];
#pragma unroll
    for (int r = 0; r < RPW; ++r) {
      const int64_t row = min(row0 + r, H - 1);
      load_row<NL>(dc + row * kb * 128, ds + row * kb, kb, g, cp, row0 + r < H, w[r], s[r]);
    }
    for (int c0 = 0; c0 < cnt; c0 += NT) {
      int qa[NT][NL][8];
      float dd[NT][NL];
      int bb[NT][NL];
      int slot[NT];
#pragma unroll
      for (int tt = 0; tt < NT; ++tt) {
        const bool ok = c0 + tt < cnt;
        slot[tt] = A.slot_list[off + min(c0 + tt, cnt - 1)];
        const int64_t sl = slot[tt];
        load_acts<NL>(A.hq + sl * A.inter, A.hd + sl * kb, A.hb + sl * kb, kb, g, cp, ok, qa[tt], dd[tt], bb[tt]);
      }
#pragma unroll
      for (int r = 0; r < RPW; ++r) {
#pragma unroll
        for (int tt = 0; tt < NT; ++tt) {
          const float v = row_dot<NL>(w[r], s[r], qa[tt], dd[tt], bb[tt]);
          if (lane == 0 && c0 + tt < cnt && row0 + r < H) A.yd[(int64_t)slot[tt] * H + row0 + r] = v;
        }
      }
    }
  }
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
  for (int j = 0; j < A.topk; ++j) {
    const int64_t s = tok * A.topk + j;
    const int e = A.topk_idx[s];
    if (e < 0 || e >= A.n_experts) continue;
    const float wj = A.topk_w[s];
    const float4 v = reinterpret_cast<const float4*>(A.yd + s * A.hidden)[c4];
    acc.x = fmaf(wj, v.x, acc.x);
    acc.y = fmaf(wj, v.y, acc.y);
    acc.z = fmaf(wj, v.z, acc.z);
    acc.w = fmaf(wj, v.w, acc.w);
  }
  reinterpret_cast<float4*>(out)[i] = acc;
}

// ---------------------------------------------------------------------------------
// Many tokens per expert (prefill-sized groups): the per-expert contraction is a dense
// int8 GEMM, run on v_mfma_i32_16x16x64_i8. A workgroup owns one task: kMT tokens of one
// active expert x kMN weight rows (x2 matrices for gate/up). Per 256-column block:
//  - the token tile's codes are staged in LDS (double-buffered, rows padded to 272 bytes
//    so the 16 lanes of an operand read hit distinct banks) with their d and bsum;
//  - each wave unpacks its 16 weight rows' nibbles into B operands (lane: row l & 15,
//    chunk 4t + (l >> 4), half h gives MFMA (t, h); the A operand takes the same 16
//    columns of the token's codes, so every product pairs matching columns);
//  - four MFMAs per 16x16 output tile accumulate sum u*q from -4*bsum (u = c + 4), i.e.
//    the exact block sum isum, and one fp32 multiply-add per output applies f32(s) * d.
// Tasks are ranked hottest expert first with token tiles innermost, so the workgroups
// that read one weight tile run together and share it through L2.
// ---------------------------------------------------------------------------------

typedef int v4i __attribute__((ext_vector_type(4)));
constexpr int kAStride = 272;

__device__ __forceinline__ v4i lds_v4i(const int8_t* p) {
  const int4 v = *reinterpret_cast<const int4*>(p);
  return v4i{v.x, v.y, v.z, v.w};
}

// One block's loads for the MFMA kernel: this thread's 64-byte quarter of a token row,
// the token's block scale and code sum, and the lane's two 16-byte code chunks (and
// scale) of each weight matrix.
template <int NMAT>
struct MfmaStage {
  v4i a0, a1, a2, a3;
  uint4 w[NMAT][2];
  uint16_t s[NMAT];
  float d;
  int bs;
};

template <int NMAT>
__device__ __forceinline__ void mfma_fetch(MfmaStage<NMAT>& st, const v4i* qrow, const float* dsrc, const int32_t* bsrc,
                                           int64_t arow, const MatRsrc (&mr)[NMAT], int wrow, int kb, int g, int b) {
  st.a0 = qrow[b * 16 + 0];
  st.a1 = qrow[b * 16 + 1];
  st.a2 = qrow[b * 16 + 2];
  st.a3 = qrow[b * 16 + 3];
  st.d = dsrc[arow * kb + b];
  st.bs = bsrc[arow * kb + b];
#pragma unroll
  for (int m = 0; m < NMAT; ++m) {
#pragma unroll
    for (int c = 0; c < 2; ++c)
      st.w[m][c] = buf_load16(mr[m].codes, (uint32_t)((wrow * kb + b) * 128 + (4 * c + g) * 16), 0);
    st.s[m] = buf_load_u16(mr[m].scales, (uint32_t)((wrow * kb + b) * 2), 0);
  }
}

template <int NMAT>  // 2: gate and up, h = SiLU(g) * u; 1: down, y per slot
__global__ __launch_bounds__(256) void k_moe_mfma(MoeArgs A) {
  __shared__ __attribute__((aligned(16))) int8_t s_a[2][kMT * kAStride];
  __shared__ __attribute__((aligned(16))) float s_d[2][kMT];
  __shared__ __attribute__((aligned(16))) int s_b[2][kMT];
  __shared__ int s_slot[kMT];
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int li = lane & 15, g = lane >> 4;
  const int K = NMAT == 2 ? A.hidden : A.inter;
  const int N = NMAT == 2 ? A.inter : A.hidden;
  const int kb = K / 256;
  const int RT = NMAT == 2 ? A.tiles_mgu : A.tiles_mdn;
  const int n_active = A.ctrl[kNActive];
  const int n_tasks = A.ctrl[NMAT == 2 ? kTasksMGU : kTasksMDn];
  const int8_t* qsrc = NMAT == 2 ? A.xq : A.hq;
  const float* dsrc = NMAT == 2 ? A.xd : A.hd;
  const int32_t* bsrc = NMAT == 2 ? A.xb : A.hb;
  const int tt = threadIdx.x >> 2, part = threadIdx.x & 3;  // staging: token row, 64-byte quarter
  for (int task = blockIdx.x; task < n_tasks; task += gridDim.x) {
    // active expert a with tt_off[a] * RT <= task < tt_off[a + 1] * RT
    int lo = 0, hi = n_active - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (A.tt_off[mid] * RT <= task) lo = mid;
      else hi = mid - 1;
    }
    const int a = lo;
    const int ntt = A.tt_off[a + 1] - A.tt_off[a];
    const int local = task - A.tt_off[a] * RT;
    const int rtile = local / ntt, ttile = local - rtile * ntt;
    const int64_t e = A.active[a];
    const int off = A.act_off[a], cnt = A.act_off[a + 1] - off;
    const int m0 = ttile * kMT, nvalid = min(kMT, cnt - m0);
    __syncthreads();  // the previous task's readers of s_slot and s_a are done
    if (threadIdx.x < kMT) s_slot[threadIdx.x] = A.slot_list[off + m0 + min((int)threadIdx.x, nvalid - 1)];
    __syncthreads();
    const int64_t arow = NMAT == 2 ? (int64_t)(s_slot[tt] / A.topk) : (int64_t)s_slot[tt];
    const v4i* qrow = reinterpret_cast<const v4i*>(qsrc + arow * K + part * 64);  // per-lane row: plain loads
    const int wrow = min(rtile * kMN + wv * 16 + li, N - 1);
    MatRsrc mr[NMAT];
#pragma unroll
    for (int m = 0; m < NMAT; ++m) {
      const int p = NMAT == 2 ? m : 2;
      mr[m] = mat_rsrc(A.codes[p] + e * A.stride_codes[p], A.scales[p] + e * A.stride_scales[p], N, kb);
    }
    float acc[4][NMAT][4];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int m = 0; m < NMAT; ++m)
#pragma unroll
        for (int v = 0; v < 4; ++v) acc[mt][m][v] = 0.0f;

    MfmaStage<NMAT> st;
    mfma_fetch<NMAT>(st, qrow, dsrc, bsrc, arow, mr, wrow, kb, g, 0);
    for (int b = 0; b < kb; ++b) {
      const int buf = b & 1;
      v4i* dst = reinterpret_cast<v4i*>(s_a[buf] + tt * kAStride + part * 64);
      dst[0] = st.a0;
      dst[1] = st.a1;
      dst[2] = st.a2;
      dst[3] = st.a3;
      if (part == 0) {
        s_d[buf][tt] = st.d;
        s_b[buf][tt] = st.bs;
      }
      uint4 wc[NMAT][2];
      float sf[NMAT];
#pragma unroll
      for (int m = 0; m < NMAT; ++m) {
        wc[m][0] = st.w[m][0];
        wc[m][1] = st.w[m][1];
        sf[m] = f16_bits_to_f32(st.s[m]);
      }
      if (b + 1 < kb) mfma_fetch<NMAT>(st, qrow, dsrc, bsrc, arow, mr, wrow, kb, g, b + 1);
      __syncthreads();
      v4i bop[NMAT][2][2];
#pragma unroll
      for (int m = 0; m < NMAT; ++m)
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const uint4 w = wc[m][c];
          bop[m][c][0] = v4i{int(w.x & kLowNibbles), int(w.y & kLowNibbles), int(w.z & kLowNibbles), int(w.w & kLowNibbles)};
          bop[m][c][1] = v4i{int((w.x >> 4) & kLowNibbles), int((w.y >> 4) & kLowNibbles), int((w.z >> 4) & kLowNibbles),
                             int((w.w >> 4) & kLowNibbles)};
        }
#pragma unroll
      for (int mt = 0; mt < 4; ++mt) {
        const int8_t* arow_lds = s_a[buf] + (mt * 16 + li) * kAStride;
        v4i aop[2][2];
#pragma unroll
        for (int c = 0; c < 2; ++c)
#pragma unroll
          for (int h = 0; h < 2; ++h) aop[c][h] = lds_v4i(arow_lds + 32 * (4 * c + g) + 16 * h);
        const int4 bs4 = *reinterpret_cast<const int4*>(&s_b[buf][mt * 16 + 4 * g]);
        const float4 d4 = *reinterpret_cast<const float4*>(&s_d[buf][mt * 16 + 4 * g]);
#pragma unroll
        for (int m = 0; m < NMAT; ++m) {
          v4i C = v4i{-4 * bs4.x, -4 * bs4.y, -4 * bs4.z, -4 * bs4.w};
          C = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop[0][0], bop[m][0][0], C, 0, 0, 0);
          C = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop[0][1], bop[m][0][1], C, 0, 0, 0);
          C = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop[1][0], bop[m][1][0], C, 0, 0, 0);
          C = __builtin_amdgcn_mfma_i32_16x16x64_i8(aop[1][1], bop[m][1][1], C, 0, 0, 0);
          acc[mt][m][0] = fmaf(sf[m] * d4.x, (float)C[0], acc[mt][m][0]);
          acc[mt][m][1] = fmaf(sf[m] * d4.y, (float)C[1], acc[mt][m][1]);
          acc[mt][m][2] = fmaf(sf[m] * d4.z, (float)C[2], acc[mt][m][2]);
          acc[mt][m][3] = fmaf(sf[m] * d4.w, (float)C[3], acc[mt][m][3]);
        }
      }
    }
    // output: token tile row mt*16 + 4g + v, weight row orow
    const int orow = rtile * kMN + wv * 16 + li;
    if (orow < N) {
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int v = 0; v < 4; ++v) {
          const int t = mt * 16 + 4 * g + v;
          if (t < nvalid) {
            const int64_t slot = s_slot[t];
            if constexpr (NMAT == 2) A.h[slot * A.inter + orow] = silu_f32(acc[mt][0][v]) * acc[mt][1][v];
            else A.yd[slot * A.hidden + orow] = acc[mt][0][v];
          }
        }
    }
  }
}

// ---------------------------------------------------------------------------------
// Single-token step (t == 1, topk <= 8): two kernels and no dispatch pass. Each slot
// is its own task (a duplicated expert is simply computed twice), so the expert comes
// straight from topk_idx; x is quantized once per workgroup into LDS while the weight
// loads are in flight; the down kernel requantizes every slot's h into LDS once per
// workgroup and folds the weighted combine into registers, in ascending slot order
// (the same fmaf chain as k_moe_combine, so both paths give identical bits).
// ---------------------------------------------------------------------------------

constexpr int kT1MaxTopk = 8;
constexpr int kT1MaxHq = 16384;  // topk * inter bytes of requantized hidden held in LDS

// Quantize 256-block `blk` of src into LDS (one block per 8-lane group): codes, the
// block scale and code sum, and each 32-column chunk's code sum (for the lanes that later
// read the chunk). `store` is group-uniform; the quantization itself runs regardless, so
// that the loads of v are not sunk into a branch behind the weight loads.
__device__ __forceinline__ void quantize_to_lds(const float (&v)[32], int blk, int cp, int8_t* s_q, float* s_d,
                                                int* s_b, int* s_qs, bool store) {
  int qw[8], qs, bs;
  float dd;
  quantize_group32(v, qw, qs, dd, bs);
  if (!store) return;
  int4* qp = reinterpret_cast<int4*>(s_q + blk * 256 + cp * 32);
  qp[0] = make_int4(qw[0], qw[1], qw[2], qw[3]);
  qp[1] = make_int4(qw[4], qw[5], qw[6], qw[7]);
  s_qs[blk * 8 + cp] = qs;
  if (cp == 0) {
    s_d[blk] = dd;
    s_b[blk] = bs;
  }
}

__device__ __forceinline__ void load32(const float* p, float (&v)[32]) {
  const float4* q = reinterpret_cast<const float4*>(p);
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const float4 f = q[m];
    v[4 * m + 0] = f.x;
    v[4 * m + 1] = f.y;
    v[4 * m + 2] = f.z;
    v[4 * m + 3] = f.w;
  }
}

// A lane's slice of one token's quantized activations, from LDS: for load i, block
// b = 8i + g, chunk cp: 32 codes, the chunk's code sum and the block scale. Blocks past
// the end of the row (ragged k) read as zero.
template <int NL>
struct LaneActs {
  int q[NL][8];
  int qs[NL];
  float d[NL];
};

template <int NL, bool RAGGED>
__device__ __forceinline__ void lds_acts(const int8_t* s_q, const float* s_d, const int* s_qs, int kb, int g, int cp,
                                         LaneActs<NL>& a) {
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int b = 8 * i + g;
    const bool v = !RAGGED || b < kb;
    const int bc = v ? b : kb - 1;
    const int4* p = reinterpret_cast<const int4*>(s_q + bc * 256 + cp * 32);
    const int4 lo = p[0], hi = p[1];
    a.q[i][0] = v ? lo.x : 0; a.q[i][1] = v ? lo.y : 0; a.q[i][2] = v ? lo.z : 0; a.q[i][3] = v ? lo.w : 0;
    a.q[i][4] = v ? hi.x : 0; a.q[i][5] = v ? hi.y : 0; a.q[i][6] = v ? hi.z : 0; a.q[i][7] = v ? hi.w : 0;
    a.qs[i] = v ? s_qs[bc * 8 + cp] : 0;
    a.d[i] = v ? s_d[bc] : 0.0f;
  }
}

// One row's lane slice in registers: NL 16-byte code chunks and their f16 scales.
template <int NL>
struct LaneRow {
  uint4 w[NL];
  uint16_t s[NL];
};

// Row `row` (wave-uniform) of a matrix: the lane's NL chunks and their scales. Chunks past
// the row end reload the row's last block (their activations are zero).
template <int NL>
__device__ __forceinline__ void load_lane_row(const MatRsrc& m, int row, int kb, int g, int cp, LaneRow<NL>& r) {
  const uint32_t srow = (uint32_t)row * (uint32_t)kb;
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const uint32_t bc = (uint32_t)min(8 * i + g, kb - 1);
    r.w[i] = buf_load16(m.codes, bc * 128u + (uint32_t)cp * 16u, srow * 128u);
    r.s[i] = buf_load_u16(m.scales, bc * 2u, srow * 2u);
  }
}

// The lane's 32 fp32 values of 256-block `blk` of a row-major fp32 buffer.
__device__ __forceinline__ void buf_load32f(__amdgpu_buffer_rsrc_t r, uint32_t blk, int cp, float (&v)[32]) {
  const uint32_t o = (blk * 256u + (uint32_t)cp * 32u) * 4u;
#pragma unroll
  for (int m = 0; m < 8; ++m) {
    const uint4 u = buf_load16(r, o + 16u * m, 0, 0);
    v[4 * m + 0] = __uint_as_float(u.x);
    v[4 * m + 1] = __uint_as_float(u.y);
    v[4 * m + 2] = __uint_as_float(u.z);
    v[4 * m + 3] = __uint_as_float(u.w);
  }
}

// The lane's contribution to one row against one token: per load, the exact integer dot
// of its 32 codes (sum u*q - 4*qs = sum c*q, |.| <= 16256) times f32(s) * d.
template <int NL>
__device__ __forceinline__ float lane_row_dot(const LaneRow<NL>& r, const LaneActs<NL>& a) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < NL; ++i) {
    const int p = dot_chunk_u(r.w[i], a.q[i]) - 4 * a.qs[i];
    acc = fmaf(f16_bits_to_f32(r.s[i]) * a.d[i], (float)p, acc);
  }
  return acc;
}

// WAVES waves per workgroup; each wave owns RPW rows (a power of two) of gate and of up
// of one slot. After the lane partials, one butterfly leaves row r's (g, u) in the lanes
// whose low bits, reversed, spell r.
template <int NL, int RPW, int WAVES, bool RAGGED>
__global__ __launch_bounds__(WAVES * 64) void k_t1_gateup(const float* __restrict__ x, MoeArgs A) {
  static_assert(RPW == 1 || RPW == 2 || RPW == 4 || RPW == 8, "RPW must be a power of two <= 8");
  __shared__ __attribute__((aligned(16))) int8_t s_q[kMaxK];
  __shared__ float s_d[kMaxK / 256];
  __shared__ int s_b[kMaxK / 256];
  __shared__ int s_qs[kMaxK / 32];
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 3, cp = lane & 7, gid = wv * 8 + g;
  const int kb = A.hidden / 256, I = A.inter;
  const int j = blockIdx.x / A.tiles_gu, tile = blockIdx.x - j * A.tiles_gu;
  const int e = A.topk_idx[j];
  const bool valid = e >= 0 && e < A.n_experts;
  const int64_t ec = valid ? e : 0;
  const int row0 = (tile * WAVES + wv) * RPW;

  // x first (its wait must not queue behind the weights), then every weight load
  const __amdgpu_buffer_rsrc_t xr = make_rsrc(x, (uint32_t)A.hidden * 4u);
  float v[32];
  buf_load32f(xr, (uint32_t)min(gid, kb - 1), cp, v);
  __builtin_amdgcn_sched_barrier(0);
  const MatRsrc mr[2] = {mat_rsrc(A.codes[0] + ec * A.stride_codes[0], A.scales[0] + ec * A.stride_scales[0], I, kb),
                         mat_rsrc(A.codes[1] + ec * A.stride_codes[1], A.scales[1] + ec * A.stride_scales[1], I, kb)};
  LaneRow<NL> wr[2 * RPW];  // [2r] gate row r, [2r + 1] up row r
#pragma unroll
  for (int r = 0; r < RPW; ++r) {
    const int row = min(row0 + r, I - 1);
#pragma unroll
    for (int m = 0; m < 2; ++m) load_lane_row<NL>(mr[m], row, kb, g, cp, wr[2 * r + m]);
  }
  quantize_to_lds(v, min(gid, kb - 1), cp, s_q, s_d, s_b, s_qs, gid < kb);
  for (int blk = gid + WAVES * 8; blk < kb; blk += WAVES * 8) {
    buf_load32f(xr, (uint32_t)blk, cp, v);
    quantize_to_lds(v, blk, cp, s_q, s_d, s_b, s_qs, true);
  }
  __syncthreads();
  if (blockIdx.x == 0) {  // stage buffers and the status word, once per call
    for (int i = threadIdx.x; i < kb * 64; i += WAVES * 64)
      reinterpret_cast<int*>(A.xq)[i] = reinterpret_cast<const int*>(s_q)[i];
    for (int i = threadIdx.x; i < kb; i += WAVES * 64) {
      A.xd[i] = s_d[i];
      A.xb[i] = s_b[i];
    }
    if (threadIdx.x == 0) {
      int bad = 0;
      for (int jj = 0; jj < A.topk; ++jj) bad |= (A.topk_idx[jj] < 0) | (A.topk_idx[jj] >= A.n_experts);
      A.ctrl[kFlags] = bad;
    }
  }
  if (!valid || row0 >= I) return;
  LaneActs<NL> act;
  lds_acts<NL, RAGGED>(s_q, s_d, s_qs, kb, g, cp, act);
  float val[2 * RPW];
#pragma unroll
  for (int m = 0; m < 2 * RPW; ++m) val[m] = lane_row_dot<NL>(wr[m], act);
  // butterfly over the row index, then plain sums over the remaining lane bits
  if constexpr (RPW >= 2) bfly_step<2 * RPW, 1>(val);
  if constexpr (RPW >= 4) bfly_step<RPW, 2>(val);
  if constexpr (RPW >= 8) bfly_step<RPW / 2, 4>(val);
#pragma unroll
  for (int m = 0; m < 2; ++m) {
    float t = val[m];
    if constexpr (RPW < 2) t = xor_sum<1>(t);
    if constexpr (RPW < 4) t = xor_sum<2>(t);
    if constexpr (RPW < 8) t = xor_sum<4>(t);
    t = xor_sum<32>(xor_sum<16>(xor_sum<8>(t)));
    val[m] = t;
  }
  // lane bits (0, 1, 2) reversed give the row this lane holds
  const int rb = RPW == 1 ? 0 : (RPW == 2 ? (lane & 1) : (RPW == 4 ? ((lane & 1) << 1) | ((lane >> 1) & 1)
                                                                    : ((lane & 1) << 2) | (lane & 2) | ((lane >> 2) & 1)));
  if (lane < RPW && row0 + rb < I) A.h[(int64_t)j * I + row0 + rb] = silu_f32(val[0]) * val[1];
}

// WAVES waves per workgroup; each wave owns RPW rows of down for every slot. Values
// m = slot * RPW + row (padded to V, a power of two) go through one butterfly; lane
// bits reversed give m. The per-slot results meet in LDS, where the row's lane forms
// out = sum_j w_j * y_j in ascending j.
template <int NL, int RPW, int TOPK, int WAVES, bool RAGGED>
__global__ __launch_bounds__(WAVES * 64) void k_t1_down(MoeArgs A, float* __restrict__ out) {
  constexpr int V = TOPK * RPW <= 2 ? 2 : (TOPK * RPW <= 4 ? 4 : (TOPK * RPW <= 8 ? 8 : (TOPK * RPW <= 16 ? 16 : 32)));
  static_assert(TOPK * RPW <= 32 && (RPW & (RPW - 1)) == 0, "down tile too large");
  __shared__ __attribute__((aligned(16))) int8_t s_hq[kT1MaxHq];
  __shared__ float s_hd[kT1MaxHq / 256];
  __shared__ int s_hb[kT1MaxHq / 256];
  __shared__ int s_qs[kT1MaxHq / 32];
  __shared__ float s_y[WAVES][32];
  const int lane = threadIdx.x & 63, wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int g = lane >> 3, cp = lane & 7, gid = wv * 8 + g;
  const int kb = A.inter / 256, H = A.hidden, I = A.inter;
  const int nblk = TOPK * kb;
  const int row0 = (blockIdx.x * WAVES + wv) * RPW;
  int64_t ej[TOPK];
  unsigned vmask = 0;
#pragma unroll
  for (int j = 0; j < TOPK; ++j) {
    const int e = A.topk_idx[j];
    const bool v = e >= 0 && e < A.n_experts;
    vmask |= (unsigned)v << j;
    ej[j] = v ? e : 0;
  }
  // this group's first block of h first (an unrouted slot's h is never written: such a
  // group loads the buffer's first block instead and skips the quantization)
  const int blk0 = min(gid, nblk - 1);
  const bool q0 = gid < nblk && ((vmask >> (blk0 / kb)) & 1);
  const __amdgpu_buffer_rsrc_t hr = make_rsrc(A.h, (uint32_t)(TOPK * I) * 4u);
  float v[32];
  buf_load32f(hr, (uint32_t)(q0 ? blk0 : 0), cp, v);
  __builtin_amdgcn_sched_barrier(0);
  LaneRow<NL> wr[TOPK][RPW];
#pragma unroll
  for (int j = 0; j < TOPK; ++j) {
    const MatRsrc mr = mat_rsrc(A.codes[2] + ej[j] * A.stride_codes[2], A.scales[2] + ej[j] * A.stride_scales[2], H, kb);
#pragma unroll
    for (int r = 0; r < RPW; ++r) load_lane_row<NL>(mr, min(row0 + r, H - 1), kb, g, cp, wr[j][r]);
  }
  quantize_to_lds(v, blk0, cp, s_hq, s_hd, s_hb, s_qs, q0);
  for (int blk = gid + WAVES * 8; blk < nblk; blk += WAVES * 8) {
    if (!((vmask >> (blk / kb)) & 1)) continue;
    buf_load32f(hr, (uint32_t)blk, cp, v);
    quantize_to_lds(v, blk, cp, s_hq, s_hd, s_hb, s_qs, true);
  }
  __syncthreads();
  if (blockIdx.x == 0) {  // stage buffers, once per call
    for (int i = threadIdx.x; i < TOPK * I / 4; i += WAVES * 64)
      if ((vmask >> (4 * i / I)) & 1) reinterpret_cast<int*>(A.hq)[i] = reinterpret_cast<const int*>(s_hq)[i];
    for (int i = threadIdx.x; i < nblk; i += WAVES * 64)
      if ((vmask >> (i / kb)) & 1) {
        A.hd[i] = s_hd[i];
        A.hb[i] = s_hb[i];
      }
  }
  if (row0 >= H) return;
  float val[V];
#pragma unroll
  for (int m = 0; m < V; ++m) val[m] = 0.0f;
#pragma unroll
  for (int j = 0; j < TOPK; ++j) {
    LaneActs<NL> act;
    lds_acts<NL, RAGGED>(s_hq + j * I, s_hd + j * kb, s_qs + j * kb * 8, kb, g, cp, act);
#pragma unroll
    for (int r = 0; r < RPW; ++r) val[j * RPW + r] = lane_row_dot<NL>(wr[j][r], act);
  }
  bfly_step<V, 1>(val);
  if constexpr (V >= 4) bfly_step<V / 2, 2>(val);
  if constexpr (V >= 8) bfly_step<V / 4, 4>(val);
  if constexpr (V >= 16) bfly_step<V / 8, 8>(val);
  if constexpr (V >= 32) bfly_step<V / 16, 16>(val);
  float t = val[0];
  if constexpr (V < 4) t = xor_sum<2>(t);
  if constexpr (V < 8) t = xor_sum<4>(t);
  if constexpr (V < 16) t = xor_sum<8>(t);
  if constexpr (V < 32) t = xor_sum<16>(t);
  t = xor_sum<32>(t);
  // lane l holds value m = bit-reverse of its low log2(V) bits
  constexpr int LB = V == 2 ? 1 : (V == 4 ? 2 : (V == 8 ? 3 : (V == 16 ? 4 : 5)));
  const int m = (int)(__builtin_bitreverse32((unsigned)lane) >> (32 - LB));
  if (lane < V) s_y[wv][m] = t;
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  if (lane < RPW && row0 + lane < H) {
    float acc = 0.0f;
#pragma unroll
    for (int j = 0; j < TOPK; ++j) {
      if (!((vmask >> j) & 1)) continue;
      const float y = s_y[wv][j * RPW + lane];
      acc = fmaf(A.topk_w[j], y, acc);
      A.yd[(int64_t)j * H + row0 + lane] = y;
    }
    out[row0 + lane] = acc;
  }
}

// ---------------------------------------------------------------------------------
// host side
// ---------------------------------------------------------------------------------

using moe_fn = void (*)(MoeArgs);

template <int NL, int RPW>
static moe_fn pick_gu_nt(int nt) {
  return nt == 1 ? k_moe_gateup<NL, 1, RPW> : k_moe_gateup<NL, 4, RPW>;
}
template <int NL, int RPW>
static moe_fn pick_dn_nt(int nt) {
  return nt == 1 ? k_moe_down<NL, 1, RPW> : k_moe_down<NL, 4, RPW>;
}

// gate/up: RPW = 4 (NL <= 2), 2 (NL <= 4), 1 otherwise; down: twice that (one matrix).
static int rpw_gu(int nl) { return nl <= 2 ? 4 : (nl <= 4 ? 2 : 1); }
static int rpw_dn(int nl) { return nl == 1 ? 8 : (nl <= 2 ? 4 : (nl <= 4 ? 2 : 1)); }

static moe_fn pick_gateup(int nl, int nt) {
  switch (nl) {
    case 1: return pick_gu_nt<1, 4>(nt);
    case 2: return pick_gu_nt<2, 4>(nt);
    case 3: return pick_gu_nt<3, 2>(nt);
    case 4: return pick_gu_nt<4, 2>(nt);
    case 5: return pick_gu_nt<5, 1>(nt);
    case 6: return pick_gu_nt<6, 1>(nt);
    case 7: return pick_gu_nt<7, 1>(nt);
    default: return pick_gu_nt<8, 1>(nt);
  }
}
static moe_fn pick_down(int nl, int nt) {
  switch (nl) {
    case 1: return pick_dn_nt<1, 8>(nt);
    case 2: return pick_dn_nt<2, 4>(nt);
    case 3: return pick_dn_nt<3, 2>(nt);
    case 4: return pick_dn_nt<4, 2>(nt);
    case 5: return pick_dn_nt<5, 1>(nt);
    case 6: return pick_dn_nt<6, 1>(nt);
    case 7: return pick_dn_nt<7, 1>(nt);
    default: return pick_dn_nt<8, 1>(nt);
  }
}

// Tile shapes of the single-token path (measured on MI355X; overridable at build time).
#ifndef TQ_T1_RPW_GU
#define TQ_T1_RPW_GU 4  // rows of gate and of up per wave
#endif
#ifndef TQ_T1_WAVES_GU
#define TQ_T1_WAVES_GU 4  // waves per gate/up workgroup
#endif
#ifndef TQ_T1_RPW_DN
#define TQ_T1_RPW_DN 2  // rows of down per wave, for every slot
#endif
#ifndef TQ_T1_WAVES_DN
#define TQ_T1_WAVES_DN 8  // waves per down workgroup
#endif
constexpr int kT1RpwGU = TQ_T1_RPW_GU;
constexpr int kT1WavesGU = TQ_T1_WAVES_GU;
constexpr int kT1RpwDn = TQ_T1_RPW_DN;
constexpr int kT1WavesDn = TQ_T1_WAVES_DN;

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

template <int NL, bool R>
static t1dn_fn pick_t1_down_k(int topk) {
  switch (topk) {
    case 1: return k_t1_down<NL, kT1RpwDn, 1, kT1WavesDn, R>;
    case 2: return k_t1_down<NL, kT1RpwDn, 2, kT1WavesDn, R>;
    case 3: return k_t1_down<NL, kT1RpwDn, 3, kT1WavesDn, R>;
    case 4: return k_t1_down<NL, kT1RpwDn, 4, kT1WavesDn, R>;
    case 5: return k_t1_down<NL, kT1RpwDn, 5, kT1WavesDn, R>;
    case 6: return k_t1_down<NL, kT1RpwDn, 6, kT1WavesDn, R>;
    case 7: return k_t1_down<NL, kT1RpwDn, 7, kT1WavesDn, R>;
    default: return k_t1_down<NL, kT1RpwDn, 8, kT1WavesDn, R>;
  }
}

// topk * inter <= 16384 bytes of LDS bounds NL: inter <= 16384 / topk.
template <bool R>
static t1dn_fn pick_t1_down_r(int nl, int topk) {
  switch (nl) {
    case 1: return pick_t1_down_k<1, R>(topk);
    case 2: return pick_t1_down_k<2, R>(topk);
    case 3: case 4: return pick_t1_down_k<4, R>(topk);
    default: return pick_t1_down_k<8, R>(topk);
  }
}
static t1dn_fn pick_t1_down(int kb, int topk) {
  const int nl = (kb + 7) / 8;
  // NL is rounded up to 4 or 8 for nl > 2: those loads may run past the row end too
  const bool ragged = kb % 8 != 0 || (nl > 2 && nl != 4 && nl != 8);
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

// A stage with no kernel of its own on this path: its event pair is recorded back to back.
static tq_status empty_stage(void* const* events, int stage, hipStream_t st, const char* fn) {
  if (!events) return TQ_OK;
  if (hipEventRecord((hipEvent_t)events[2 * stage], st) != hipSuccess ||
      hipEventRecord((hipEvent_t)events[2 * stage + 1], st) != hipSuccess)
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

static tq_status moe_run(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                         const float* topk_w, int32_t topk, float* out, void* ws, size_t ws_bytes, int32_t flags,
                         void* stream, void* const* events, const char* fn) {
  clear_error();
  tq_status st = validate_experts(ex, fn);
  if (st != TQ_OK) return st;
  if (t < 0 || t > (1 << 20)) return fail(TQ_ERR_INVALID, "%s: t = %lld outside [0, 2^20]", fn, (long long)t);
  if (topk < 1 || topk > kMaxTopk || topk > ex->n_experts)
    return fail(TQ_ERR_INVALID, "%s: topk = %d outside [1, min(%d, n_experts)]", fn, topk, kMaxTopk);
  if (flags & ~(TQ_MOE_FORCE_VALU | TQ_MOE_FORCE_MFMA) || flags == (TQ_MOE_FORCE_VALU | TQ_MOE_FORCE_MFMA))
    return fail(TQ_ERR_INVALID, "%s: bad flags 0x%x", fn, flags);
  if (t == 0) {
    for (int i = 0; i < kNumStages; ++i)
      if ((st = empty_stage(events, i, (hipStream_t)stream, fn)) != TQ_OK) return st;
    return TQ_OK;
  }
  if (!x || !topk_idx || !topk_w || !out || !ws) return fail(TQ_ERR_INVALID, "%s: null pointer", fn);
  if (!aligned(x, 16) || !aligned(out, 16) || !aligned(ws, 256) || !aligned(topk_idx, 4) || !aligned(topk_w, 4))
    return fail(TQ_ERR_ALIGN, "%s: x and out must be 16-byte aligned, ws 256-byte aligned", fn);
  const Layout L = make_layout(ex->n_experts, ex->hidden, ex->inter, t, topk);
  if (ws_bytes < L.total)
    return fail(TQ_ERR_WORKSPACE, "%s: workspace %zu bytes < required %zu", fn, ws_bytes, L.total);

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
  A.slot_list = reinterpret_cast<int32_t*>(base + L.slot_list);
  A.xq = reinterpret_cast<int8_t*>(base + L.xq);
  A.xd = reinterpret_cast<float*>(base + L.xd);
  A.xb = reinterpret_cast<int32_t*>(base + L.xb);
  A.h = reinterpret_cast<float*>(base + L.h);
  A.hq = reinterpret_cast<int8_t*>(base + L.hq);
  A.hd = reinterpret_cast<float*>(base + L.hd);
  A.hb = reinterpret_cast<int32_t*>(base + L.hb);
  A.yd = reinterpret_cast<float*>(base + L.yd);

  const int nl_gu = (ex->hidden / 256 + 7) / 8, nl_dn = (ex->inter / 256 + 7) / 8;
  const int nt = t == 1 ? 1 : 4;
  A.tiles_gu = (ex->inter + 4 * rpw_gu(nl_gu) - 1) / (4 * rpw_gu(nl_gu));
  A.tiles_dn = (ex->hidden + 4 * rpw_dn(nl_dn) - 1) / (4 * rpw_dn(nl_dn));
  const int64_t S = t * topk;
  const int64_t max_active = std::min<int64_t>(S, ex->n_experts);
  const int64_t cap = 256 * 16;  // workgroups per launch; the rest are strided over them
  const unsigned g_gu = (unsigned)std::min<int64_t>(max_active * A.tiles_gu, cap);
  const unsigned g_dn = (unsigned)std::min<int64_t>(max_active * A.tiles_dn, cap);
  const int64_t xblocks = t * (ex->hidden / 256), hblocks = S * (ex->inter / 256);
  const int nq = (int)((xblocks + 31) / 32);
  hipStream_t stm = (hipStream_t)stream;

  (void)hipGetLastError();
  if (t == 1 && topk <= kT1MaxTopk && (int64_t)topk * ex->inter <= kT1MaxHq && !(flags & TQ_MOE_FORCE_MFMA)) {
    // single token: gate_up, then down with the requant and the combine fused; the
    // prologue, requant and combine stages are empty on this path
    const int rgu = t1_rpw_gu(nl_gu);
    A.tiles_gu = (ex->inter + kT1WavesGU * rgu - 1) / (kT1WavesGU * rgu);
    const unsigned tiles_dn = (unsigned)((ex->hidden + kT1WavesDn * kT1RpwDn - 1) / (kT1WavesDn * kT1RpwDn));
    if ((st = empty_stage(events, 0, stm, fn)) != TQ_OK) return st;
    if ((st = launch_stage(events, 1, pick_t1_gateup(ex->hidden / 256), dim3((unsigned)(topk * A.tiles_gu)), kT1WavesGU * 64, stm,
                           fn, x, A)) != TQ_OK)
      return st;
    if ((st = empty_stage(events, 2, stm, fn)) != TQ_OK) return st;
    if ((st = launch_stage(events, 3, pick_t1_down(ex->inter / 256, topk), dim3(tiles_dn), kT1WavesDn * 64, stm, fn, A, out)) !=
        TQ_OK)
      return st;
    return empty_stage(events, 4, stm, fn);
  }
  // per-expert contraction on MFMA for prefill-sized groups (or when forced), VALU dot4
  // otherwise
  const bool mfma = (flags & TQ_MOE_FORCE_MFMA) || (!(flags & TQ_MOE_FORCE_VALU) && S >= kMfmaMinSlots);
  A.tiles_mgu = (ex->inter + kMN - 1) / kMN;
  A.tiles_mdn = (ex->hidden + kMN - 1) / kMN;
  const int64_t max_tiles = S / kMT + max_active;
  const unsigned g_mgu = (unsigned)std::min<int64_t>(max_tiles * A.tiles_mgu, cap);
  const unsigned g_mdn = (unsigned)std::min<int64_t>(max_tiles * A.tiles_mdn, cap);
  if ((st = launch_stage(events, 0, k_moe_prologue, dim3(nq + 1), 256, stm, fn, x, A, nq)) != TQ_OK) return st;
  if (mfma) st = launch_stage(events, 1, k_moe_mfma<2>, dim3(g_mgu), 256, stm, fn, A);
  else st = launch_stage(events, 1, pick_gateup(nl_gu, nt), dim3(g_gu), 256, stm, fn, A);
  if (st != TQ_OK) return st;
  if ((st = launch_stage(events, 2, k_moe_requant, dim3((unsigned)((hblocks + 31) / 32)), 256, stm, fn, A, hblocks)) !=
      TQ_OK)
    return st;
  if (mfma) st = launch_stage(events, 3, k_moe_mfma<1>, dim3(g_mdn), 256, stm, fn, A);
  else st = launch_stage(events, 3, pick_down(nl_dn, nt), dim3(g_dn), 256, stm, fn, A);
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
  return TQ_OK;
}

extern "C" tq_status tq_moe_grouped(const tq_experts* ex, const float* x, int64_t t, const int32_t* topk_idx,
                                    const float* topk_w, int32_t topk, float* out, void* ws, size_t ws_bytes,
                                    int32_t flags, void* stream) {
  return tq::moe_run(ex, x, t, topk_idx, topk_w, topk, out, ws, ws_bytes, flags, stream, nullptr, "tq_moe_grouped");
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
  e = hipMemcpy(flags_out, static_cast<const uint8_t*>(ws) + L.ctrl + 4 * kFlags, 4, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return fail(TQ_ERR_DEVICE, "tq_moe_status: copy failed: %s", hipGetErrorString(e));
  return TQ_OK;
}
