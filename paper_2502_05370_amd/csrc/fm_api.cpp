// Host layer of libfinemoe_map: argument validation, store handles, buffer
// layout and dispatch to the kernels.  Every entry point validates all of its
// arguments before enqueueing anything and reports failures as an fm_status
// plus a thread-local message; no C++ exception crosses the ABI.
#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <mutex>
#include <new>
#include <string>

#include "fm_internal.h"

namespace {

thread_local std::string g_error;

fm_status fail(fm_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_error = buf;
  return st;
}

fm_status ok() {
  g_error.clear();
  return FM_OK;
}

fm_status hip_fail(hipError_t e, const char* what) {
  return fail(FM_ERR_HIP, "%s: %s (%d)", what, hipGetErrorString(e), static_cast<int>(e));
}

size_t elem_size(fm_dtype t) { return t == FM_BF16 ? 2 : 4; }

bool valid_dtype(int t) { return t == FM_F32 || t == FM_BF16; }

constexpr size_t kMaxGroupBytes = 0xF0000000u;

struct Layout {
  size_t plane_bytes, maps, rnorm, embs, norms, flags, total;
  int64_t plane_elems;
};

// Buffer layout: [L map planes][L prefix inverse-norm planes][embeddings]
// [embedding norms][flags], 256-byte aligned parts.
bool make_layout(int32_t cap, int32_t L, int32_t E, int32_t d_emb, fm_dtype t, Layout* out) {
  if (cap < 1 || L < 1 || E < 1 || d_emb < 0 || !valid_dtype(t)) return false;
  Layout ly;
  const size_t es = elem_size(t);
  ly.plane_bytes = fm::align_up(static_cast<size_t>(fm::round16(cap)) * fm::row_elems(E) * es, fm::kAlign);
  ly.plane_elems = static_cast<int64_t>(ly.plane_bytes / es);
  ly.maps = ly.plane_bytes * L;
  ly.rnorm = fm::align_up(static_cast<size_t>(fm::rnorm_stride(cap)) * L * 4, fm::kAlign);
  ly.embs = fm::align_up(static_cast<size_t>(fm::round16(cap)) * d_emb * 2, fm::kAlign);
  ly.norms = d_emb > 0 ? fm::align_up(static_cast<size_t>(cap) * 4, fm::kAlign) : 0;
  ly.flags = fm::kAlign;
  ly.total = ly.maps + ly.rnorm + ly.embs + ly.norms + ly.flags;
  *out = ly;
  return true;
}

}  // namespace

struct fm_store {
  fm::StoreView v;
  int device;
};

namespace {

fm_status check_workspace(const fm_store* s, void* ws, size_t bytes) {
  if (ws == nullptr) return fail(FM_ERR_INVALID, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % fm::kAlign != 0)
    return fail(FM_ERR_INVALID, "workspace must be %zu-byte aligned", fm::kAlign);
  const size_t need = fm::workspace_bytes_needed(s->v.L, s->v.E, s->v.d_emb, s->v.map_dtype);
  if (bytes < need) return fail(FM_ERR_INVALID, "workspace of %zu bytes is smaller than the %zu bytes required", bytes, need);
  return FM_OK;
}

fm::Workspace carve(const fm_store*, void* ws) { return fm::carve_workspace(ws); }

}  // namespace

namespace fm {

ScanEvents& scan_events() {
  thread_local ScanEvents ev;
  return ev;
}

// Workspace layout: [partial][perm][sdep][rq][pgrp][rgrp][ngrp][qrows], each part 256-byte
// aligned.  qrows holds the staged queries of one launch: the trajectory
// planes, or the tiled semantic queries (1024 x d_emb bf16).

// Parts before the staged queries (partial lists, positions, groups).
static size_t workspace_fixed_bytes() {
  size_t b = align_up(sizeof(uint64_t) * kChunkB * kMaxPartials * kMaxK, kAlign);
  b += 3 * align_up(sizeof(int32_t) * kChunkB, kAlign);
  b += 3 * align_up(sizeof(int32_t) * (kChunkB / 16), kAlign);
  return b;
}

size_t workspace_bytes_needed(int32_t L, int32_t E, int32_t d_emb, fm_dtype map_dtype) {
  const size_t traj = traj_qrows_bytes(L, E, map_dtype, kChunkB);
  const size_t sem = static_cast<size_t>(kChunkB) * d_emb * 2;
  return workspace_fixed_bytes() + align_up(traj > sem ? traj : sem, kAlign);
}

// What a trajectory search alone reads and writes of a workspace.
size_t workspace_bytes_trajectory(int32_t L, int32_t E, fm_dtype map_dtype) {
  return workspace_fixed_bytes() + align_up(traj_qrows_bytes(L, E, map_dtype, kChunkB), kAlign);
}

Workspace carve_workspace(void* base) {
  char* p = static_cast<char*>(base);
  Workspace w;
  w.partial = reinterpret_cast<uint64_t*>(p);
  p += align_up(sizeof(uint64_t) * kChunkB * kMaxPartials * kMaxK, kAlign);
  w.perm = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * kChunkB, kAlign);
  w.sdep = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * kChunkB, kAlign);
  w.rq = reinterpret_cast<float*>(p);
  p += align_up(sizeof(float) * kChunkB, kAlign);
  w.pgrp = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (kChunkB / 16), kAlign);
  w.rgrp = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (kChunkB / 16), kAlign);
  w.ngrp = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * (kChunkB / 16), kAlign);
  w.qrows = p;
  return w;
}

}  // namespace fm

namespace {

fm_status check_store(const fm_store* s) {
  if (s == nullptr) return fail(FM_ERR_INVALID, "store handle is NULL");
  return FM_OK;
}

fm_status check_workspace(const fm_store* s, void* ws, size_t bytes);

// The kernels run on the store's device; make it current for the enqueue.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) {
      ok = false;
      return;
    }
    if (prev != dev && hipSetDevice(dev) != hipSuccess) ok = false;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

}  // namespace

extern "C" {

int32_t fm_version(void) { return (1 << 16) | 0; }

const char* fm_last_error(void) { return g_error.c_str(); }

size_t fm_map_bytes(int32_t cap, int32_t L, int32_t E, fm_dtype map_dtype) {
  Layout ly;
  if (!make_layout(cap, L, E, 0, map_dtype, &ly)) return 0;
  return ly.maps;
}

size_t fm_store_bytes(int32_t cap, int32_t L, int32_t E, int32_t d_emb, fm_dtype map_dtype) {
  Layout ly;
  if (!make_layout(cap, L, E, d_emb, map_dtype, &ly)) return 0;
  return ly.total;
}

size_t fm_workspace_bytes(int32_t L, int32_t E, int32_t d_emb, fm_dtype map_dtype, int32_t B_max, int32_t k_max) {
  if (L < 1 || L > fm::kMaxL || E < 1 || E > fm::kMaxE || !valid_dtype(map_dtype)) return 0;
  if (d_emb < 0 || d_emb % 128 != 0) return 0;
  if (B_max < 1 || k_max < 1 || k_max > fm::kMaxK) return 0;
  return fm::workspace_bytes_needed(L, E, d_emb, map_dtype);
}

fm_status fm_store_build(fm_store** out, const fm_store_desc* d) {
  if (out == nullptr || d == nullptr) return fail(FM_ERR_INVALID, "out and desc must be non-NULL");
  if (!valid_dtype(d->map_dtype)) return fail(FM_ERR_INVALID, "map_dtype %d is not FM_F32 or FM_BF16", d->map_dtype);
  if (d->cap < 1 || d->L < 1 || d->E < 1 || d->d_emb < 0)
    return fail(FM_ERR_INVALID, "cap=%d L=%d E=%d d_emb=%d out of range", d->cap, d->L, d->E, d->d_emb);
  if (d->E > fm::kMaxE) return fail(FM_ERR_UNSUPPORTED, "E=%d exceeds %d experts per layer", d->E, fm::kMaxE);
  if (d->L > fm::kMaxL) return fail(FM_ERR_UNSUPPORTED, "L=%d exceeds %d layers", d->L, fm::kMaxL);
  if (d->d_emb % 128 != 0)
    return fail(FM_ERR_UNSUPPORTED, "d_emb=%d is not a multiple of 128", d->d_emb);
  if (fm::round16(d->cap) * fm::row_elems(d->E) > (static_cast<int64_t>(1) << 31) - 1)
    return fail(FM_ERR_UNSUPPORTED, "cap*E exceeds 2^31-1");
  Layout ly;
  make_layout(d->cap, d->L, d->E, d->d_emb, d->map_dtype, &ly);
  // The trajectory scan addresses one group of up to 32/E layer planes with
  // 32-bit byte offsets.
  const size_t group_planes = (d->E >= 8 && 32 % d->E == 0) ? static_cast<size_t>(32 / d->E) : 1;
  if (ly.plane_bytes * group_planes > kMaxGroupBytes)
    return fail(FM_ERR_UNSUPPORTED, "cap=%d: %zu bytes per layer group of map planes exceed %zu", d->cap,
                ly.plane_bytes * group_planes, kMaxGroupBytes);
  // ... and the prefix inverse norms of all layers with 32-bit byte offsets.
  if (static_cast<size_t>(d->L) * static_cast<size_t>(fm::rnorm_stride(d->cap)) * 4 > kMaxGroupBytes)
    return fail(FM_ERR_UNSUPPORTED, "cap=%d L=%d: the prefix inverse norms exceed %zu bytes", d->cap, d->L,
                kMaxGroupBytes);
  if (d->buffer == nullptr) return fail(FM_ERR_INVALID, "buffer is NULL");
  if (reinterpret_cast<uintptr_t>(d->buffer) % fm::kAlign != 0)
    return fail(FM_ERR_INVALID, "buffer must be %zu-byte aligned", fm::kAlign);
  if (d->buffer_bytes < ly.total)
    return fail(FM_ERR_INVALID, "buffer of %zu bytes is smaller than fm_store_bytes = %zu", d->buffer_bytes, ly.total);
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  fm_store* s = new (std::nothrow) fm_store;
  if (s == nullptr) return fail(FM_ERR_INVALID, "out of host memory");
  char* base = static_cast<char*>(d->buffer);
  s->v.planes = base;
  s->v.plane_elems = ly.plane_elems;
  s->v.rnorm = reinterpret_cast<float*>(base + ly.maps);
  s->v.rn_stride = fm::rnorm_stride(d->cap);
  char* after = base + ly.maps + ly.rnorm;
  s->v.embs = d->d_emb > 0 ? reinterpret_cast<uint16_t*>(after) : nullptr;
  s->v.emb_norm = d->d_emb > 0 ? reinterpret_cast<float*>(after + ly.embs) : nullptr;
  s->v.flags = reinterpret_cast<uint32_t*>(after + ly.embs + ly.norms);
  s->v.cap = d->cap;
  s->v.L = d->L;
  s->v.E = d->E;
  s->v.row = fm::row_elems(d->E);
  s->v.d_emb = d->d_emb;
  s->v.n = 0;
  s->v.map_dtype = d->map_dtype;
  s->device = dev;
  // Clear the device flags once (synchronous, outside any stream work).
  e = hipMemset(s->v.flags, 0, fm::kAlign);
  if (e != hipSuccess) {
    delete s;
    return hip_fail(e, "hipMemset(flags)");
  }
  *out = s;
  return ok();
}

fm_status fm_store_insert(fm_store* s, const void* maps, const void* embs, int32_t n, int32_t* slots_out,
                          void* stream) {
  if (fm_status st = check_store(s)) return st;
  if (n < 0) return fail(FM_ERR_INVALID, "n=%d is negative", n);
  if (n == 0) return ok();
  if (maps == nullptr) return fail(FM_ERR_INVALID, "maps is NULL");
  if (s->v.d_emb > 0 && embs == nullptr) return fail(FM_ERR_INVALID, "store has d_emb=%d but embs is NULL", s->v.d_emb);
  if (s->v.d_emb > 0 && reinterpret_cast<uintptr_t>(embs) % 16 != 0)
    return fail(FM_ERR_INVALID, "embs must be 16-byte aligned");
  if (static_cast<int64_t>(s->v.n) + n > s->v.cap)
    return fail(FM_ERR_FULL, "inserting %d into a store holding %d of %d", n, s->v.n, s->v.cap);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_insert(s->v, maps, embs, n, nullptr, slots_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "insert launch");
  s->v.n += n;
  return ok();
}

size_t fm_dedup_scratch_bytes(int32_t cap, int32_t n_max) {
  if (cap < 1 || n_max < 1 || n_max > fm::kChunkB) return 0;
  return fm::dedup_scratch_bytes(cap, n_max);
}

fm_status fm_store_insert_dedup(fm_store* s, const void* maps, const void* embs, int32_t n, int32_t d,
                                int32_t* slots_out, void* ws, size_t ws_bytes, void* scratch, size_t scratch_bytes,
                                void* stream) {
  if (fm_status st = check_store(s)) return st;
  if (n < 0 || n > fm::kChunkB) return fail(FM_ERR_INVALID, "n=%d outside [0, %d]", n, fm::kChunkB);
  if (n == 0) return ok();
  if (maps == nullptr) return fail(FM_ERR_INVALID, "maps is NULL");
  if (d < 0 || d > s->v.L) return fail(FM_ERR_INVALID, "prefetch distance d=%d outside [0, L=%d]", d, s->v.L);
  if (d > 0 && s->v.d_emb == 0)
    return fail(FM_ERR_INVALID, "prefetch distance d=%d weighs semantic scores but the store has no embeddings", d);
  if (s->v.d_emb > 0 && embs == nullptr) return fail(FM_ERR_INVALID, "store has d_emb=%d but embs is NULL", s->v.d_emb);
  if (s->v.d_emb > 0 && reinterpret_cast<uintptr_t>(embs) % 16 != 0)
    return fail(FM_ERR_INVALID, "embs must be 16-byte aligned");
  if (fm_status st = check_workspace(s, ws, ws_bytes)) return st;
  if (scratch == nullptr) return fail(FM_ERR_INVALID, "scratch is NULL");
  if (reinterpret_cast<uintptr_t>(scratch) % fm::kAlign != 0)
    return fail(FM_ERR_INVALID, "scratch must be %zu-byte aligned", fm::kAlign);
  const size_t need = fm::dedup_scratch_bytes(s->v.cap, n);
  if (scratch_bytes < need)
    return fail(FM_ERR_INVALID, "scratch of %zu bytes is smaller than fm_dedup_scratch_bytes(cap=%d, n=%d) = %zu",
                scratch_bytes, s->v.cap, n, need);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  const fm::DedupScratch sc = fm::carve_dedup_scratch(scratch, s->v.cap, n);
  hipError_t e = fm::launch_insert_dedup(s->v, maps, embs, n, d, slots_out, carve(s, ws), sc,
                                         static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "deduplicating insert launch");
  const int32_t room = s->v.cap - s->v.n;
  s->v.n += n < room ? n : room;
  return ok();
}

fm_status fm_store_size(const fm_store* s, int32_t* n_out) {
  if (fm_status st = check_store(s)) return st;
  if (n_out == nullptr) return fail(FM_ERR_INVALID, "n_out is NULL");
  *n_out = s->v.n;
  return ok();
}

fm_status fm_store_check(fm_store* s, void* stream, uint32_t* flags_out) {
  if (fm_status st = check_store(s)) return st;
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipStream_t st = static_cast<hipStream_t>(stream);
  uint32_t flags = 0;
  hipError_t e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  e = hipMemcpy(&flags, s->v.flags, sizeof(flags), hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy(flags)");
  e = hipMemset(s->v.flags, 0, sizeof(uint32_t));
  if (e != hipSuccess) return hip_fail(e, "hipMemset(flags)");
  if (flags_out != nullptr) *flags_out = flags;
  if (flags != 0)
    return fail(FM_ERR_DEVICE, "device flags 0x%x (1: depth clamped, 2: index out of range, 4: stale step state)", flags);
  return ok();
}

fm_status fm_store_destroy(fm_store* s) {
  if (fm_status st = check_store(s)) return st;
  delete s;
  return ok();
}

static fm_status check_match_common(const fm_store* s, int32_t B, int32_t k, const int32_t* idx_out,
                                    const float* score_out, void* ws, size_t ws_bytes) {
  if (fm_status st = check_store(s)) return st;
  if (B < 1 || B > 65536) return fail(FM_ERR_INVALID, "B=%d outside [1, 65536]", B);
  if (k < 1 || k > fm::kMaxK) return fail(FM_ERR_INVALID, "k=%d outside [1, %d]", k, fm::kMaxK);
  if (idx_out == nullptr || score_out == nullptr) return fail(FM_ERR_INVALID, "idx_out and score_out must be non-NULL");
  return check_workspace(s, ws, ws_bytes);
}

// The selection's own arguments (Section 4.3 parameters, layer ranges, outputs).
static fm_status check_select(const fm_store* s, const int32_t* lb, const int32_t* le, const fm_select_params* p,
                              const uint64_t* mask_out, const uint8_t* count_out) {
  if (lb == nullptr || le == nullptr || p == nullptr || mask_out == nullptr || count_out == nullptr)
    return fail(FM_ERR_INVALID, "layer_begin, layer_end, params, mask_out and count_out must be non-NULL");
  if (p->mode != FM_TAU_FIXED && p->mode != FM_TAU_DYNAMIC) return fail(FM_ERR_INVALID, "tau mode %d", p->mode);
  if (p->blend != FM_BLEND_NONE && p->blend != FM_BLEND_SCORE) return fail(FM_ERR_INVALID, "blend %d", p->blend);
  if (p->k_min < 0 || p->k_min > p->k_max || p->k_max > s->v.E)
    return fail(FM_ERR_INVALID, "need 0 <= k_min (%d) <= k_max (%d) <= E (%d)", p->k_min, p->k_max, s->v.E);
  if (p->mode == FM_TAU_FIXED && p->tau != p->tau) return fail(FM_ERR_INVALID, "tau is NaN");
  return FM_OK;
}

fm_status fm_match_semantic(const fm_store* s, const void* q, int32_t B, int32_t k, int32_t* idx_out,
                            float* score_out, void* ws, size_t ws_bytes, void* stream) {
  if (fm_status st = check_match_common(s, B, k, idx_out, score_out, ws, ws_bytes)) return st;
  if (q == nullptr) return fail(FM_ERR_INVALID, "q is NULL");
  if (reinterpret_cast<uintptr_t>(q) % 16 != 0) return fail(FM_ERR_INVALID, "q must be 16-byte aligned");
  if (s->v.d_emb == 0) return fail(FM_ERR_INVALID, "store has no embeddings (d_emb = 0)");
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_match_semantic(s->v, q, B, k, idx_out, score_out, nullptr, carve(s, ws),
                                           static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "semantic match launch");
  return ok();
}

fm_status fm_match_trajectory(const fm_store* s, const void* q, const int32_t* depth, int32_t max_depth,
                              int32_t B, int32_t k, int32_t* idx_out, float* score_out, void* ws,
                              size_t ws_bytes, void* stream) {
  if (fm_status st = check_match_common(s, B, k, idx_out, score_out, ws, ws_bytes)) return st;
  if (q == nullptr || depth == nullptr) return fail(FM_ERR_INVALID, "q and depth must be non-NULL");
  if (max_depth < 1 || max_depth > s->v.L)
    return fail(FM_ERR_INVALID, "max_depth=%d outside [1, L=%d]", max_depth, s->v.L);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_match_trajectory(s->v, q, depth, max_depth, B, k, idx_out, score_out, nullptr,
                                             carve(s, ws), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "trajectory match launch");
  return ok();
}

fm_status fm_miss_count(const fm_store* s, const void* q, int32_t B, int32_t K, const uint64_t* masks,
                        const int32_t* lb, const int32_t* le, uint8_t* miss_out, void* stream) {
  if (fm_status st = check_store(s)) return st;
  if (q == nullptr || masks == nullptr || lb == nullptr || le == nullptr || miss_out == nullptr)
    return fail(FM_ERR_INVALID, "q, masks, layer_begin, layer_end and miss_out must be non-NULL");
  if (B < 1 || B > 65536) return fail(FM_ERR_INVALID, "B=%d outside [1, 65536]", B);
  if (K < 1 || K > s->v.E) return fail(FM_ERR_INVALID, "K=%d outside [1, E=%d]", K, s->v.E);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_miss(s->v, q, B, K, masks, lb, le, miss_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "miss count launch");
  return ok();
}

fm_status fm_priority_order(const fm_store* s, const int32_t* idx, const float* score, int32_t B, int32_t k,
                            fm_blend blend, fm_pri_kind kind, const uint64_t* masks, const int32_t* l_now,
                            const float* freq, int32_t cap, int32_t* order_out, float* pri_out, int32_t* count_out,
                            void* stream) {
  if (fm_status st = check_store(s)) return st;
  if (idx == nullptr || score == nullptr || masks == nullptr || order_out == nullptr || pri_out == nullptr ||
      count_out == nullptr)
    return fail(FM_ERR_INVALID, "idx, score, masks, order_out, pri_out and count_out must be non-NULL");
  if (B < 1 || B > 65536) return fail(FM_ERR_INVALID, "B=%d outside [1, 65536]", B);
  if (k < 1 || k > fm::kMaxK) return fail(FM_ERR_INVALID, "k=%d outside [1, %d]", k, fm::kMaxK);
  if (blend != FM_BLEND_NONE && blend != FM_BLEND_SCORE) return fail(FM_ERR_INVALID, "blend %d", blend);
  if (kind != FM_PRI_PREFETCH && kind != FM_PRI_EVICT) return fail(FM_ERR_INVALID, "priority kind %d", kind);
  if (kind == FM_PRI_PREFETCH && l_now == nullptr) return fail(FM_ERR_INVALID, "l_now is NULL");
  if (kind == FM_PRI_EVICT && freq == nullptr) return fail(FM_ERR_INVALID, "freq is NULL");
  if (cap < 1 || cap > fm::kMaxL * fm::kMaxE) return fail(FM_ERR_INVALID, "cap=%d outside [1, %d]", cap, fm::kMaxL * fm::kMaxE);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_priority(s->v, idx, score, B, k, blend, kind, masks, l_now, freq, cap, order_out,
                                     pri_out, count_out, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "priority launch");
  return ok();
}

size_t fm_traj_state_bytes(int32_t cap, int32_t B_max) {
  if (cap < 1 || B_max < 1 || B_max > 65536) return 0;
  return fm::traj_state_bytes(cap, B_max);
}

fm_status fm_traj_step(fm_store* s, void* state, size_t state_bytes, const void* q, int32_t layer, int32_t B,
                       int32_t k, int32_t* idx_out, float* score_out, void* ws, size_t ws_bytes, void* stream) {
  if (fm_status st = check_match_common(s, B, k, idx_out, score_out, ws, ws_bytes)) return st;
  if (q == nullptr) return fail(FM_ERR_INVALID, "q_layer is NULL");
  if (layer < 0 || layer >= s->v.L) return fail(FM_ERR_INVALID, "layer=%d outside [0, L=%d)", layer, s->v.L);
  if (state == nullptr) return fail(FM_ERR_INVALID, "state is NULL");
  if (reinterpret_cast<uintptr_t>(state) % fm::kAlign != 0)
    return fail(FM_ERR_INVALID, "state must be %zu-byte aligned", fm::kAlign);
  const size_t need = fm::traj_state_bytes(s->v.cap, B);
  if (state_bytes < need)
    return fail(FM_ERR_INVALID, "state of %zu bytes is smaller than fm_traj_state_bytes(cap=%d, B=%d) = %zu",
                state_bytes, s->v.cap, B, need);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_traj_step(s->v, state, q, layer, B, k, idx_out, score_out, carve(s, ws),
                                      static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "trajectory step launch");
  return ok();
}

fm_status fm_select_prefetch(const fm_store* s, const int32_t* idx, const float* score, int32_t B, int32_t k,
                             const int32_t* lb, const int32_t* le, const fm_select_params* p,
                             uint64_t* mask_out, uint8_t* count_out, void* stream) {
  if (fm_status st = check_store(s)) return st;
  if (idx == nullptr || score == nullptr) return fail(FM_ERR_INVALID, "idx and score must be non-NULL");
  if (B < 1 || B > 65536) return fail(FM_ERR_INVALID, "B=%d outside [1, 65536]", B);
  if (k < 1 || k > fm::kMaxK) return fail(FM_ERR_INVALID, "k=%d outside [1, %d]", k, fm::kMaxK);
  if (fm_status st = check_select(s, lb, le, p, mask_out, count_out)) return st;
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipError_t e = fm::launch_select(s->v, idx, score, B, k, lb, le, *p, mask_out, count_out,
                                   static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "select launch");
  return ok();
}

fm_status fm_match_semantic_select(const fm_store* s, const void* q, int32_t B, int32_t k, const int32_t* lb,
                                   const int32_t* le, const fm_select_params* p, int32_t* idx_out, float* score_out,
                                   uint64_t* mask_out, uint8_t* count_out, void* ws, size_t ws_bytes,
                                   void* stream) {
  if (fm_status st = check_match_common(s, B, k, idx_out, score_out, ws, ws_bytes)) return st;
  if (q == nullptr) return fail(FM_ERR_INVALID, "q is NULL");
  if (reinterpret_cast<uintptr_t>(q) % 16 != 0) return fail(FM_ERR_INVALID, "q must be 16-byte aligned");
  if (s->v.d_emb == 0) return fail(FM_ERR_INVALID, "store has no embeddings (d_emb = 0)");
  if (fm_status st = check_select(s, lb, le, p, mask_out, count_out)) return st;
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  const fm::SelectFuse fuse{lb, le, *p, mask_out, count_out};
  hipError_t e = fm::launch_match_semantic(s->v, q, B, k, idx_out, score_out, nullptr, carve(s, ws),
                                           static_cast<hipStream_t>(stream), nullptr, 1.0, 0.0, &fuse);
  if (e != hipSuccess) return hip_fail(e, "semantic match-and-select launch");
  return ok();
}

fm_status fm_match_trajectory_select(const fm_store* s, const void* q, const int32_t* depth, int32_t max_depth,
                                     int32_t B, int32_t k, const int32_t* lb, const int32_t* le,
                                     const fm_select_params* p, int32_t* idx_out, float* score_out,
                                     uint64_t* mask_out, uint8_t* count_out, void* ws, size_t ws_bytes,
                                     void* stream) {
  if (fm_status st = check_match_common(s, B, k, idx_out, score_out, ws, ws_bytes)) return st;
  if (q == nullptr || depth == nullptr) return fail(FM_ERR_INVALID, "q and depth must be non-NULL");
  if (max_depth < 1 || max_depth > s->v.L)
    return fail(FM_ERR_INVALID, "max_depth=%d outside [1, L=%d]", max_depth, s->v.L);
  if (fm_status st = check_select(s, lb, le, p, mask_out, count_out)) return st;
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  const fm::SelectFuse fuse{lb, le, *p, mask_out, count_out};
  hipError_t e = fm::launch_match_trajectory(s->v, q, depth, max_depth, B, k, idx_out, score_out, nullptr,
                                             carve(s, ws), static_cast<hipStream_t>(stream), &fuse);
  if (e != hipSuccess) return hip_fail(e, "trajectory match-and-select launch");
  return ok();
}

fm_status fm_debug_scores(const fm_store* s, const void* q, const int32_t* depth, int32_t max_depth,
                          const void* q_sem, int32_t B, float* scores_out, void* ws, size_t ws_bytes,
                          void* stream) {
  if (fm_status st = check_store(s)) return st;
  if ((q == nullptr) == (q_sem == nullptr)) return fail(FM_ERR_INVALID, "exactly one of q and q_sem must be non-NULL");
  if (B < 1 || B > 65536) return fail(FM_ERR_INVALID, "B=%d outside [1, 65536]", B);
  if (scores_out == nullptr) return fail(FM_ERR_INVALID, "scores_out is NULL");
  if (fm_status st = check_workspace(s, ws, ws_bytes)) return st;
  if (s->v.n == 0) return ok();
  // Same kernels as the match calls; only the dense score output is written.
  fm::Workspace w = carve(s, ws);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  hipStream_t st = static_cast<hipStream_t>(stream);
  hipError_t e;
  if (q != nullptr) {
    if (depth == nullptr) return fail(FM_ERR_INVALID, "depth is NULL");
    if (max_depth < 1 || max_depth > s->v.L)
      return fail(FM_ERR_INVALID, "max_depth=%d outside [1, L=%d]", max_depth, s->v.L);
    e = fm::launch_match_trajectory(s->v, q, depth, max_depth, B, 1, nullptr, nullptr, scores_out, w, st);
  } else {
    if (s->v.d_emb == 0) return fail(FM_ERR_INVALID, "store has no embeddings (d_emb = 0)");
    e = fm::launch_match_semantic(s->v, q_sem, B, 1, nullptr, nullptr, scores_out, w, st);
  }
  if (e != hipSuccess) return hip_fail(e, "debug scores launch");
  return ok();
}

// ---------------------------------------------------------------- allocation-free trajectory search

}  // extern "C"

namespace {

// Workspace of fm_match_trajectory_noalloc: a device array of the library.
// Each GPU it runs on holds its own copy until the process ends.  Host code
// never passes the array's name to a kernel or a copy (on the host it only
// stands in for the symbol); it uses the device address looked up once per
// device by scratch_address().
constexpr size_t kScratchBytes = FM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on device dev, which must be current.
fm_status scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return fail(FM_ERR_UNSUPPORTED, "device %d beyond %d devices", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (ptr == nullptr || reinterpret_cast<uintptr_t>(ptr) % fm::kAlign != 0)
      return fail(FM_ERR_HIP, "device scratch at %p is not %zu-byte aligned", ptr, fm::kAlign);
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return FM_OK;
}

}  // namespace

extern "C" {

fm_status fm_match_trajectory_noalloc(const fm_store* s, const void* q, const int32_t* depth, int32_t max_depth,
                                      int32_t B, int32_t k, int32_t* idx_out, float* score_out, void* stream) {
  if (fm_status st = check_store(s)) return st;
  if (B < 1 || B > 65536) return fail(FM_ERR_INVALID, "B=%d outside [1, 65536]", B);
  if (k < 1 || k > fm::kMaxK) return fail(FM_ERR_INVALID, "k=%d outside [1, %d]", k, fm::kMaxK);
  if (idx_out == nullptr || score_out == nullptr) return fail(FM_ERR_INVALID, "idx_out and score_out must be non-NULL");
  if (q == nullptr || depth == nullptr) return fail(FM_ERR_INVALID, "q and depth must be non-NULL");
  if (max_depth < 1 || max_depth > s->v.L)
    return fail(FM_ERR_INVALID, "max_depth=%d outside [1, L=%d]", max_depth, s->v.L);
  const size_t need = fm::workspace_bytes_trajectory(s->v.L, s->v.E, s->v.map_dtype);
  if (need > kScratchBytes)
    return fail(FM_ERR_UNSUPPORTED, "a trajectory search of L=%d x E=%d needs %zu bytes of workspace, beyond the %zu "
                "bytes of the library's device scratch", s->v.L, s->v.E, need, kScratchBytes);
  DeviceGuard dg(s->device);
  if (!dg.ok) return fail(FM_ERR_HIP, "cannot select the store's device %d", s->device);
  void* ws = nullptr;
  if (fm_status st = scratch_address(s->device, &ws)) return st;
  hipError_t e = fm::launch_match_trajectory(s->v, q, depth, max_depth, B, k, idx_out, score_out, nullptr,
                                             fm::carve_workspace(ws), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "trajectory match launch");
  return ok();
}

fm_status fm_debug_scan_events(void* start, void* stop) {
  if ((start == nullptr) != (stop == nullptr)) return fail(FM_ERR_INVALID, "start and stop must both be set or both NULL");
  fm::scan_events().start = static_cast<hipEvent_t>(start);
  fm::scan_events().stop = static_cast<hipEvent_t>(stop);
  return ok();
}

}  // extern "C"
