// Internal interfaces between the C-ABI layer and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "saga.h"

namespace saga {

// counters kept at plan->counts
enum Count : int {
  kNumSegments = 0,
  kNumBlocks = 1,
  kNSplit = 2,
  kSSplit = 3,
  kErrFlags = 4,
  kMaxDegree = 5,
  kCountSlots = 8
};
// error bits in counts[kErrFlags]: 1, 2, 4, 8 are CSR errors (see saga.h);
// this one marks a broken internal invariant of the plan builder
constexpr int kErrInternal = 1 << 16;

// ---- plan.hip ----
struct PlanLayout {
  size_t off_d_in, off_d_out, off_perm, off_first, off_seg_row, off_seg_beg, off_seg_end,
      off_block_ptr, off_counts, off_scratch, scratch_bytes, total;
  int64_t max_segments, max_blocks, max_split, max_split_segments;
  int64_t radix_tiles, scan_tiles_rows, scan_tiles_segs;
  int64_t outdeg_nb, edge_tiles;
  bool outdeg_bucketed;
};

bool plan_layout(int32_t num_dst, int32_t num_src, int64_t num_edges, int32_t seg_len,
                 int32_t block_cost, int32_t row_cost, PlanLayout* L);

// order_st, fork, join: see saga_plan_build_split (all null: one stream)
hipError_t launch_plan_build(const saga_plan& p, const PlanLayout& L, hipStream_t st,
                             hipStream_t order_st = nullptr, hipEvent_t fork = nullptr,
                             hipEvent_t join = nullptr);

// ---- gather.hip ----
struct GatherArgs {
  // plan
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* d_in;
  const int32_t* d_out;
  const int32_t* perm;
  const int32_t* row_seg_first;
  const int32_t* seg_row;
  const int32_t* seg_beg;
  const int32_t* seg_end;
  const int32_t* block_ptr;
  const int32_t* counts;
  int64_t max_blocks;
  int64_t max_split;
  int block_cost;  // the plan's row-block cost
  int bpw;         // row blocks per workgroup (set by the launchers; >= 1)
  // op
  int msg, reduce, dtype, heads, head_mean, dst_norm, act;
  float neg_slope;
  int feat;        // F (input feature columns)
  int out_cols;    // F or F/heads
  // inputs
  const void* src; int64_t ld_src;
  int64_t src_rows;  // rows of src (sizes the slices run per launch)
  const float* el; int64_t ld_el;
  const float* er; int64_t ld_er;
  const float* gsrc; int64_t ld_gsrc;
  const float* gdst; int64_t ld_gdst;
  const float* efeat; int64_t ld_efeat; int fe;
  const float* w_edge;
  const float* gate_bias;
  const float* bias;
  // output
  void* out; int64_t ld_out;
  // split-row partials (float32), stride pstride floats per segment
  float* partial; int64_t pstride;
  int pcols;       // partial accumulator columns; softmax m/l follow at pcols
  int identity;    // source row of edge e is row e (unfused segment reduction)
  // typed messages: source row of CSR entry e is col_idx[e] (= the rel
  // plan's edge_pair), scaled by edge_scale[e]; err2: the rel plan's flags
  const float* edge_scale;
  const int32_t* err2;
  // added to every output row before the bias (nullable; dtype of out)
  const void* self; int64_t ld_self;
  // fused next transform (xn > 0): the Gather's output h (in `out`, a
  // workspace) is multiplied as rows finish: xout[v] = xrs(v) * (h_v xw),
  // xw F x xn (dtype), columns from xsplit on (xsplit > 0) going to xtail
  const void* xw; int xn; int xsplit;
  // xw packed as W^T for the matrix cores (workspace): 16 * ceil(xn / 16)
  // rows of xldwt 16-byte vectors (F columns, zero rows past xn, a 16-byte
  // pad per row)
  uint4* xwt; int xldwt;
  void* xout; int64_t ld_xout;
  void* xtail; int64_t ld_xtail;
  const int32_t* xrs;
};

int gather_partial_cols(int64_t feat);
size_t gather_partial_stride(const saga_edge_op& op, int64_t feat);
hipError_t launch_gather(const GatherArgs& a, hipStream_t st);
// the fused Gather + next transform (COPY with SUM or MEAN, whole 128-byte
// slices, at most four of them, xn <= 64); xf_pack_bytes: the packed W^T
int64_t xf_pack_bytes(int64_t feat, int esize, int xn);
hipError_t launch_gather_transform(const GatherArgs& a, hipStream_t st);
// unfused baseline: materialise msg (E x ldm, CSR order), then reduce it
hipError_t launch_unfused(const GatherArgs& a, int64_t E, void* msg, int64_t ldm, hipStream_t st);

// ---- gemm.hip ----
struct GemmArgs {
  int dtype, mode, act;
  int64_t M, N, K, K2;
  const void* a; int64_t lda;
  const void* w; int64_t ldw;
  const void* a2; int64_t lda2;
  const void* w2; int64_t ldw2;
  const float* bias;
  const float* bias2;
  const int32_t* row_scale_deg;
  void* out; int64_t ldo;
  // split output: columns >= split go to out2 (ld ldo2) at column c - split
  int64_t split; void* out2; int64_t ldo2;
  // scratch for the packed transposed weights (gemm_workspace_bytes)
  void* ws; size_t ws_bytes;
  // set by launch_gemm: packed weights in the workspace, ld kp / kp2
  const void* wt; int64_t kp;
  const void* wt2; int64_t kp2;
  // grouped mode (launch_gemm_grouped): row q of A is row arow[q] of a (a
  // negative entry gives an all-zero output row); w holds `groups` K x N
  // weights stacked; rows [grp_ptr[g], grp_ptr[g+1]) use weight g, ranges
  // are whole tiles, grp_ptr[groups] is the row count; err1 / err2 nonzero:
  // do nothing
  const int32_t* arow;
  const int32_t* grp_ptr;
  int groups;
  int64_t wt_group_stride;
  const int32_t* err1;
  const int32_t* err2;
};
// LSTM Gather (GraphSAGE): recurrence over each row's in-edges
struct LstmArgs {
  const int32_t* row_ptr;
  const int32_t* col_idx;
  const int32_t* perm;
  const int32_t* counts;
  int32_t num_dst;
  int hidden;                          // H: 32, 64 or 128
  const float* gates_x; int64_t ld_gx; // num_src x 4H: x W_ih + b_ih + b_hh
  const float* w_hh; int64_t ld_whh;   // H x 4H
  float* out; int64_t ld_out;          // num_dst x H
  int32_t* queue;                      // work-queue counter (workspace)
  int32_t perm_begin, perm_end;        // rows at these perm positions
};
hipError_t launch_lstm_gather(const LstmArgs& a, hipStream_t st);

// bytes of workspace launch_gemm needs for these shapes (packed weights)
size_t gemm_workspace_bytes(int dtype, int mode, int64_t N, int64_t K, int64_t K2);
hipError_t launch_gemm(const GemmArgs& g, hipStream_t st);
// grouped GEMM over row ranges of whole kRelTile-row tiles (mode ignored;
// M = row capacity, a multiple of kRelTile)
size_t gemm_grouped_workspace_bytes(int dtype, int groups, int64_t N, int64_t K);
hipError_t launch_gemm_grouped(const GemmArgs& g, hipStream_t st);

// ---- rel.hip ----
constexpr int kRelTile = SAGA_REL_TILE;  // rows per grouped-GEMM tile
constexpr int kRelMaxRelations = SAGA_REL_MAX_RELATIONS;
enum RelCount : int { kRelRows = 0, kRelPairs = 1, kRelErr = 2, kRelCountSlots = 4 };
struct RelLayout {
  int64_t wp;        // bitmap words per relation (whole counting blocks)
  int64_t bpr;       // counting blocks per relation
  int64_t nblocks;   // counting blocks in all
  int64_t max_pairs;
  size_t off_rel_ptr, off_rel_count, off_pair_src, off_edge_pair, off_edge_norm, off_counts,
      off_scratch, off_bitmap, off_word_base, off_bcnt, off_block_base, scratch_bytes, total;
  bool use_flags;    // byte flags packed into the bitmap (else bitmap atomics)
  size_t off_flags;
};
bool rel_layout(int32_t num_src, int64_t num_edges, int32_t num_rel, RelLayout* L);
hipError_t launch_rel_build(const saga_plan& p, const saga_rel_plan& rel, const RelLayout& L,
                            hipStream_t st);

// ---- layer helpers (gather.hip) ----
hipError_t launch_fold_attention(const float* w, int64_t K, int64_t F, int heads, const float* al,
                                 const float* ar, float* w_ext, int64_t ld_ext, hipStream_t st);

}  // namespace saga
