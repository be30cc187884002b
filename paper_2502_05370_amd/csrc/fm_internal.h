// Internal declarations shared by the host layer and the kernel sources of
// libfinemoe_map.  Not part of the public ABI (include/finemoe_map.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "finemoe_map.h"

namespace fm {

constexpr int kMaxL = 64;            // layers per map
constexpr int kMaxE = 64;            // experts per layer (mask width)
constexpr int kMaxK = 8;             // matches kept per query
constexpr int kChunkB = 1024;        // queries per scan launch
constexpr int kMaxPartials = 256;    // partial top-k lists per query (workgroups per query group)
constexpr size_t kAlign = 256;

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Map planes are tiled: plane l holds the maps in tiles of 16 consecutive maps;
// inside a tile, each quad of 4 consecutive experts (e = 4q .. 4q+3) stores
// the 16 maps' 4 values contiguously, so one wave reading 4 quads of a tile
// reads one contiguous block.  row = E rounded up to a multiple of 4 (the
// padding is stored as zeros), so a tile holds 16 * row elements.
inline int32_t row_elems(int32_t E) { return (E + 3) / 4 * 4; }
inline int64_t round16(int64_t cap) { return (cap + 15) / 16 * 16; }
__host__ __device__ __forceinline__ int64_t tile_offset(int64_t y, int32_t e, int32_t row) {
  return (y / 16) * 16 * row + (e / 4) * 64 + (y % 16) * 4 + (e % 4);
}
// Embeddings (and staged semantic queries) are tiled as MFMA operands: for a
// block of 16 rows and a k-step of 32 dimensions, a contiguous 1 KB tile holds
// at 16-byte slot 16g + c the dimensions 32s + 8g .. +7 of row c (the operand
// of lane 16g + c of v_mfma_f32_16x16x32_bf16).  d is a multiple of 128.
__host__ __device__ __forceinline__ int64_t emb_offset(int64_t y, int32_t e, int32_t d) {
  return ((y / 16) * (d / 32) + e / 32) * 512 + (16 * ((e % 32) / 8) + y % 16) * 8 + (e % 8);
}
// Stride of the prefix inverse-norm planes: cap rounded up to 64 maps.
inline int64_t rnorm_stride(int32_t cap) { return (static_cast<int64_t>(cap) + 63) / 64 * 64; }

// Device view of a store: layer-major map planes, prefix inverse norms,
// embeddings and their norms.
struct StoreView {
  void* planes;          // [L] tiled planes (tile_offset) of map dtype; plane stride plane_elems
  int64_t plane_elems;   // elements per plane (round16(cap) * row, padded to 256 bytes)
  float* rnorm;          // [L][rn_stride]: 1/|x[y][0:l+1]| (0 for a zero prefix, NaN for NaN)
  int64_t rn_stride;
  uint16_t* embs;        // round16(cap) x d_emb bf16, tiled (emb_offset)
  float* emb_norm;       // [cap]
  uint32_t* flags;       // sticky FM_FLAG_* bits
  int32_t cap, L, E, row, d_emb, n;
  fm_dtype map_dtype;
};

// Match workspace of one launch (every part is fully rewritten by the
// launch that reads it, so it needs no initialisation).
struct Workspace {
  uint64_t* partial;  // [kChunkB][kMaxPartials][kMaxK] per-workgroup top-k keys
  int32_t* perm;      // [kChunkB] query index at each depth-sorted position (-1: padding)
  int32_t* sdep;      // [kChunkB] clamped depth at each position (0: padding)
  float* rq;          // [kChunkB] 1/|query prefix| at each position
  int32_t* pgrp;      // [kChunkB / 16] first scan workgroup of each query group (trajectory)
  int32_t* rgrp;      // [kChunkB / 16] scan workgroups (partial lists) of each query group
  int32_t* ngrp;      // [kChunkB / 16] layer groups each query group's scan walks
  void* qrows;        // staged query rows of every layer group (trajectory)
};
size_t workspace_bytes_needed(int32_t L, int32_t E, int32_t d_emb, fm_dtype map_dtype);
size_t workspace_bytes_trajectory(int32_t L, int32_t E, fm_dtype map_dtype);

// Scratch of a deduplicating insert: [depth][slots][cand][cand_score] sized
// for kChunkB new iterations, then the two dense score matrices of n_max x
// cap float32 (each part 256-byte aligned).  Rewritten by every call.
struct DedupScratch {
  int32_t* depth;       // [kChunkB] full depth L for the trajectory scan
  int32_t* slots;       // [kChunkB] slot of each new iteration (-1: dropped)
  int32_t* cand;        // [kChunkB][8] best replacement candidates
  float* cand_score;    // [kChunkB][8] their RDY
  float* rdy;           // [m][size] RDY (or the one weighted score when d is 0 or L)
  float* traj;          // [m][size] full-depth trajectory scores (0 < d < L)
};
size_t dedup_scratch_bytes(int32_t cap, int32_t n_max);
DedupScratch carve_dedup_scratch(void* base, int32_t cap, int32_t n_max);
Workspace carve_workspace(void* base);
size_t traj_qrows_bytes(int L, int E, fm_dtype dt, int b_pad);
// partial holds R lists per position; with rgrp set, position pos merges only
// the first rgrp[pos / qg] of them.
hipError_t launch_finalize(const uint64_t* partial, const int32_t* perm, int32_t B, int32_t R, int32_t k, int KTOP,
                           int32_t* idx_out, float* score_out, hipStream_t st, const int32_t* rgrp = nullptr,
                           int32_t qg = 0);

// Caller-provided events bracketing the next scan launches on this thread
// (both null when unset); see fm_debug_scan_events.
struct ScanEvents {
  hipEvent_t start = nullptr;
  hipEvent_t stop = nullptr;
};
ScanEvents& scan_events();

// Launchers (return hipSuccess or the first HIP error).
hipError_t launch_insert(const StoreView& s, const void* maps, const void* embs, int32_t n_new,
                         const int32_t* slot_of, int32_t* slots_out, hipStream_t st);
hipError_t launch_insert_dedup(const StoreView& s, const void* maps, const void* embs, int32_t n, int32_t d,
                               int32_t* slots_out, const Workspace& ws, const DedupScratch& sc, hipStream_t st);
// The selection a fused match-and-select call runs after the merge: the
// rows' layer ranges, the parameters and the outputs, in the match call's
// batch order (pointers to its first query).
struct SelectFuse {
  const int32_t* lb;
  const int32_t* le;
  fm_select_params p;
  uint64_t* mask_out;   // [B][L]
  uint8_t* count_out;   // [B][L]
  SelectFuse at(int32_t b0, int32_t L) const {
    SelectFuse f = *this;
    f.lb = lb + b0;
    f.le = le + b0;
    f.mask_out = mask_out + static_cast<int64_t>(b0) * L;
    f.count_out = count_out + static_cast<int64_t>(b0) * L;
    return f;
  }
};
// k_finalize and k_select in one launch (fm_select.hip): the merge of the
// partial lists of positions 0 .. B-1 (query perm[pos], or pos), the
// matches written to idx_out / score_out, then each row's selection.
hipError_t launch_merge_select(const StoreView& s, const uint64_t* partial, const int32_t* perm, int32_t B, int32_t R,
                               int32_t k, int KTOP, const int32_t* rgrp, int32_t qg, int32_t* idx_out,
                               float* score_out, const SelectFuse& f, hipStream_t st);
// With fuse set, the merge of each launch is the merge-and-select above.
hipError_t launch_match_trajectory(const StoreView& s, const void* q, const int32_t* depth,
                                   int32_t max_depth, int32_t B, int32_t k, int32_t* idx_out,
                                   float* score_out, float* dbg_scores, const Workspace& ws,
                                   hipStream_t st, const SelectFuse* fuse = nullptr);
// With dbg_scores set, the dense scores are written there; with mix also set
// (a dense [B][n] matrix), the dense output is w_self * score + w_mix * mix.
hipError_t launch_match_semantic(const StoreView& s, const void* q, int32_t B, int32_t k,
                                 int32_t* idx_out, float* score_out, float* dbg_scores,
                                 const Workspace& ws, hipStream_t st, const float* mix = nullptr,
                                 double w_self = 1.0, double w_mix = 0.0, const SelectFuse* fuse = nullptr);
// Top-1 semantic scan (fm_sem_mm.hip): queries per group for a chunk of Bc
// queries, and the scan itself on queries already staged by k_sem_prep
// (b_pad = groups * queries per group); *R_out receives the partial lists per
// query for k_finalize.  The dense form (dbg set) writes every cosine, or
// w_self * cosine + w_mix * mix[b][y] when mix is set.
int sem_mm_group(int32_t Bc);
hipError_t launch_sem_mm(const StoreView& s, int32_t Bc, int32_t b_pad, const Workspace& ws, float* dbg, int32_t* R_out,
                         hipStream_t st, const float* mix = nullptr, double w_self = 1.0, double w_mix = 0.0);
// Top-1 trajectory scan of bf16 stores (fm_traj_mm.hip): whether a chunk of
// Bc queries takes it, its queries per group, and the scan itself on queries
// staged by k_traj_prep in its tiled layout (b_pad = groups * queries per
// group); *R_out receives the partial lists per query for k_finalize.
bool traj_mm_fits(bool bf, int KTOP, int32_t Bc, int32_t max_depth, int nlg, int ksg);
int traj_mm_group();
int traj_mm_workgroups();
hipError_t launch_traj_mm(const StoreView& s, int spl, int lpg, int ksg, int nlg, int32_t max_depth, int32_t b_pad,
                          const Workspace& ws, float* dbg, int32_t* R_out, hipStream_t st);
hipError_t launch_miss(const StoreView& s, const void* q, int32_t B, int32_t K, const uint64_t* masks,
                       const int32_t* lb, const int32_t* le, uint8_t* miss_out, hipStream_t st);
hipError_t launch_priority(const StoreView& s, const int32_t* idx, const float* score, int32_t B, int32_t k,
                           int32_t blend, int32_t kind, const uint64_t* masks, const int32_t* l_now,
                           const float* freq, int32_t cap, int32_t* order_out, float* pri_out, int32_t* count_out,
                           hipStream_t st);
size_t traj_state_bytes(int32_t cap, int32_t B_max);
hipError_t launch_traj_step(const StoreView& s, void* state, const void* q, int32_t layer, int32_t B, int32_t k,
                            int32_t* idx_out, float* score_out, const Workspace& ws, hipStream_t st);
hipError_t launch_select(const StoreView& s, const int32_t* idx, const float* score, int32_t B,
                         int32_t k, const int32_t* lb, const int32_t* le,
                         const fm_select_params& p, uint64_t* mask_out, uint8_t* count_out,
                         hipStream_t st);

}  // namespace fm
