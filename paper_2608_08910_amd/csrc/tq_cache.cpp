// Host-tier expert streaming (Sec. 2.2: the folded planes are the stored file itself, so
// fetching a missing expert projection costs a single contiguous read, and serving from
// HBM or from the host tier runs the same kernels on the same bytes: outputs do not
// depend on where an expert was cached; the paper's serving stack keeps pinned RAM and LRU slots in front of the file).
//
// On MI355X the tiers are pinned host memory (every expert) and a pool of expert slots
// in HBM. Each expert is one contiguous record, so a miss is one host-to-device copy; a
// slot pool of records is described to the MoE kernels as an ordinary expert stack
// (stride = record size), with the step's routing remapped from expert ids to slots.
#include <cstring>

#include "tq_internal.hpp"

namespace {

struct RecordLayout {
  int64_t codes[3], scales[3], bytes;
};

// gate, up, down codes, then gate, up, down scales; every piece 128-byte aligned.
RecordLayout record_layout(int32_t hidden, int32_t inter) {
  RecordLayout L{};
  const int64_t H = hidden, I = inter;
  const int64_t cb[3] = {I * H / 2, I * H / 2, H * I / 2};
  const int64_t sb[3] = {I * (H / 256) * 2, I * (H / 256) * 2, H * (I / 256) * 2};
  int64_t off = 0;
  for (int p = 0; p < 3; ++p) {
    L.codes[p] = off;
    off += (cb[p] + 127) / 128 * 128;
  }
  for (int p = 0; p < 3; ++p) {
    L.scales[p] = off;
    off += (sb[p] + 127) / 128 * 128;
  }
  L.bytes = off;
  return L;
}

bool shape_ok(int32_t hidden, int32_t inter) {
  return hidden >= 256 && inter >= 256 && hidden % 256 == 0 && inter % 256 == 0 && hidden <= tq::kMaxK &&
         inter <= tq::kMaxK;
}

// Planner state in a caller-owned host buffer.
struct CacheHeader {
  int32_t n_experts, n_slots;
  int64_t clock;  // advances on every map call
  uint64_t magic;
};
constexpr uint64_t kCacheMagic = 0x7471636163686531ull;

struct CacheView {
  CacheHeader* h;
  int32_t* slot_expert;  // [n_slots], -1 if empty
  int64_t* slot_last;    // [n_slots], clock of the last step that used the slot (-1 never)
  int32_t* expert_slot;  // [n_experts], -1 if not resident
  int64_t* expert_seen;  // [n_experts], clock of the last call that listed the expert
};

CacheView view(void* state, int32_t n_experts, int32_t n_slots) {
  CacheView v;
  auto* p = static_cast<uint8_t*>(state);
  v.h = reinterpret_cast<CacheHeader*>(p);
  p += sizeof(CacheHeader);
  v.slot_last = reinterpret_cast<int64_t*>(p);
  p += sizeof(int64_t) * n_slots;
  v.expert_seen = reinterpret_cast<int64_t*>(p);
  p += sizeof(int64_t) * n_experts;
  v.slot_expert = reinterpret_cast<int32_t*>(p);
  p += sizeof(int32_t) * n_slots;
  v.expert_slot = reinterpret_cast<int32_t*>(p);
  return v;
}

size_t state_bytes(int32_t n_experts, int32_t n_slots) {
  return sizeof(CacheHeader) + (sizeof(int64_t) + sizeof(int32_t)) * ((size_t)n_slots + (size_t)n_experts);
}

}  // namespace

extern "C" size_t tq_expert_record_bytes(int32_t hidden, int32_t inter) {
  if (!shape_ok(hidden, inter)) return 0;
  return (size_t)record_layout(hidden, inter).bytes;
}

extern "C" tq_status tq_experts_from_records(const void* base, int32_t n_records, int32_t hidden, int32_t inter,
                                             tq_experts* out) {
  using namespace tq;
  clear_error();
  if (!shape_ok(hidden, inter))
    return fail(TQ_ERR_INVALID, "tq_experts_from_records: hidden=%d inter=%d must be multiples of 256 in [256, %d]",
                hidden, inter, kMaxK);
  if (n_records < 1) return fail(TQ_ERR_INVALID, "tq_experts_from_records: n_records = %d < 1", n_records);
  if (!base || !out) return fail(TQ_ERR_INVALID, "tq_experts_from_records: null pointer");
  if (!aligned(base, 128)) return fail(TQ_ERR_ALIGN, "tq_experts_from_records: base must be 128-byte aligned");
  const RecordLayout L = record_layout(hidden, inter);
  const uint8_t* b = static_cast<const uint8_t*>(base);
  out->n_experts = n_records;
  out->hidden = hidden;
  out->inter = inter;
  out->gate_codes = b + L.codes[0];
  out->up_codes = b + L.codes[1];
  out->down_codes = b + L.codes[2];
  out->gate_scales = reinterpret_cast<const uint16_t*>(b + L.scales[0]);
  out->up_scales = reinterpret_cast<const uint16_t*>(b + L.scales[1]);
  out->down_scales = reinterpret_cast<const uint16_t*>(b + L.scales[2]);
  for (int p = 0; p < 3; ++p) {
    out->stride_codes[p] = L.bytes;
    out->stride_scales[p] = L.bytes / 2;
  }
  return TQ_OK;
}

extern "C" size_t tq_cache_state_bytes(int32_t n_experts, int32_t n_slots) {
  if (n_experts < 1 || n_slots < 1) return 0;
  return state_bytes(n_experts, n_slots);
}

extern "C" tq_status tq_cache_init(void* state, int32_t n_experts, int32_t n_slots) {
  using namespace tq;
  clear_error();
  if (n_experts < 1 || n_slots < 1)
    return fail(TQ_ERR_INVALID, "tq_cache_init: n_experts = %d and n_slots = %d must be >= 1", n_experts, n_slots);
  if (!state) return fail(TQ_ERR_INVALID, "tq_cache_init: null state");
  if (!aligned(state, 8)) return fail(TQ_ERR_ALIGN, "tq_cache_init: state must be 8-byte aligned");
  CacheView v = view(state, n_experts, n_slots);
  v.h->n_experts = n_experts;
  v.h->n_slots = n_slots;
  v.h->clock = 0;
  v.h->magic = kCacheMagic;
  for (int32_t s = 0; s < n_slots; ++s) {
    v.slot_expert[s] = -1;
    v.slot_last[s] = -1;
  }
  for (int32_t e = 0; e < n_experts; ++e) {
    v.expert_slot[e] = -1;
    v.expert_seen[e] = -1;
  }
  return TQ_OK;
}

extern "C" tq_status tq_cache_map(void* state, const int32_t* ids, int64_t n, int32_t* slots_out, int32_t* misses_out,
                                  int32_t* n_miss_out) {
  using namespace tq;
  clear_error();
  if (!state || (n > 0 && (!ids || !slots_out || !misses_out)) || !n_miss_out)
    return fail(TQ_ERR_INVALID, "tq_cache_map: null pointer");
  if (n < 0) return fail(TQ_ERR_INVALID, "tq_cache_map: n = %lld < 0", (long long)n);
  auto* h = static_cast<CacheHeader*>(state);
  if (h->magic != kCacheMagic) return fail(TQ_ERR_INVALID, "tq_cache_map: state was not initialized by tq_cache_init");
  CacheView v = view(state, h->n_experts, h->n_slots);
  const int64_t now = ++h->clock;
  // the step's distinct experts (marked with this call's clock)
  int64_t distinct = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int32_t e = ids[i];
    if (e < 0 || e >= h->n_experts)
      return fail(TQ_ERR_INVALID, "tq_cache_map: expert id %d at %lld out of [0, %d)", e, (long long)i, h->n_experts);
    if (v.expert_seen[e] != now) {
      v.expert_seen[e] = now;
      ++distinct;
    }
  }
  if (distinct > h->n_slots)
    return fail(TQ_ERR_INVALID, "tq_cache_map: the step needs %lld distinct experts but the pool has %d slots",
                (long long)distinct, h->n_slots);
  // from here on the call succeeds: pin the resident experts of the step
  for (int64_t i = 0; i < n; ++i) {
    const int32_t s = v.expert_slot[ids[i]];
    if (s >= 0) v.slot_last[s] = now;
  }
  // place the others, in order of first appearance: an empty slot (lowest index) first,
  // else the least recently used slot not used by this step (lowest index on ties)
  int32_t nm = 0;
  for (int64_t i = 0; i < n; ++i) {
    const int32_t e = ids[i];
    if (v.expert_slot[e] >= 0) continue;
    int32_t best = -1;
    for (int32_t s = 0; s < h->n_slots; ++s) {
      if (v.slot_last[s] >= now) continue;
      if (v.slot_expert[s] < 0) {
        best = s;
        break;
      }
      if (best < 0 || v.slot_last[s] < v.slot_last[best]) best = s;
    }
    // best >= 0: at most n_slots distinct experts are pinned in this call
    if (v.slot_expert[best] >= 0) v.expert_slot[v.slot_expert[best]] = -1;
    v.slot_expert[best] = e;
    v.slot_last[best] = now;
    v.expert_slot[e] = best;
    misses_out[2 * nm] = e;
    misses_out[2 * nm + 1] = best;
    ++nm;
  }
  for (int64_t i = 0; i < n; ++i) slots_out[i] = v.expert_slot[ids[i]];
  *n_miss_out = nm;
  return TQ_OK;
}

extern "C" tq_status tq_cache_fetch(const void* state, const void* host_store, void* dev_slots, size_t record_bytes,
                                    const int32_t* misses, int32_t n_miss, const int32_t* slots_host,
                                    int32_t* slots_dev, int64_t n, void* stream) {
  using namespace tq;
  clear_error();
  if (!state) return fail(TQ_ERR_INVALID, "tq_cache_fetch: null state");
  const auto* h = static_cast<const CacheHeader*>(state);
  if (h->magic != kCacheMagic) return fail(TQ_ERR_INVALID, "tq_cache_fetch: state was not initialized by tq_cache_init");
  if (n_miss < 0 || n < 0) return fail(TQ_ERR_INVALID, "tq_cache_fetch: negative count");
  if (record_bytes == 0 || record_bytes % 128 != 0)
    return fail(TQ_ERR_INVALID, "tq_cache_fetch: record_bytes = %zu must be a positive multiple of 128", record_bytes);
  if ((n_miss > 0 && (!host_store || !dev_slots || !misses)) || (n > 0 && (!slots_host || !slots_dev)))
    return fail(TQ_ERR_INVALID, "tq_cache_fetch: null pointer");
  (void)hipGetLastError();
  for (int32_t m = 0; m < n_miss; ++m) {
    const int64_t e = misses[2 * m], s = misses[2 * m + 1];
    if (e < 0 || e >= h->n_experts || s < 0 || s >= h->n_slots)
      return fail(TQ_ERR_INVALID, "tq_cache_fetch: miss %d names expert %lld / slot %lld outside the store or pool", m,
                  (long long)e, (long long)s);
  }
  for (int64_t i = 0; i < n; ++i)
    if (slots_host[i] < 0 || slots_host[i] >= h->n_slots)
      return fail(TQ_ERR_INVALID, "tq_cache_fetch: slot %d at %lld outside the pool", slots_host[i], (long long)i);
  const auto* src = static_cast<const uint8_t*>(host_store);
  auto* dst = static_cast<uint8_t*>(dev_slots);
  for (int32_t m = 0; m < n_miss; ++m) {
    const int64_t e = misses[2 * m], s = misses[2 * m + 1];
    const hipError_t err = hipMemcpyAsync(dst + s * (int64_t)record_bytes, src + e * (int64_t)record_bytes, record_bytes,
                                          hipMemcpyHostToDevice, (hipStream_t)stream);
    if (err != hipSuccess) return fail(TQ_ERR_DEVICE, "tq_cache_fetch: %s", hipGetErrorString(err));
  }
  if (n > 0) {
    const hipError_t err =
        hipMemcpyAsync(slots_dev, slots_host, sizeof(int32_t) * (size_t)n, hipMemcpyHostToDevice, (hipStream_t)stream);
    if (err != hipSuccess) return fail(TQ_ERR_DEVICE, "tq_cache_fetch: %s", hipGetErrorString(err));
  }
  return TQ_OK;
}
