// C-ABI entry points: argument validation, workspace carving and dispatch
// to the kernel launchers; whole-layer composition of the Table I models.
#include <hip/hip_runtime.h>
#include <rocprofiler-sdk-roctx/roctx.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <exception>
#include <mutex>
#include <vector>

#include "saga.h"
#include "saga_internal.h"

namespace {

thread_local char g_err[512] = "";

saga_status fail(saga_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return s;
}

saga_status ok() {
  g_err[0] = 0;
  return SAGA_OK;
}

saga_status dev_fail(hipError_t e, const char* where) {
  return fail(SAGA_EDEVICE, "%s: %s", where, hipGetErrorString(e));
}

inline size_t esize(int32_t t) { return t == SAGA_BF16 ? 2 : 4; }
inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }
inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

bool range_overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + nb && b0 < a0 + na;
}

size_t mat_bytes(int64_t rows, int64_t cols, int64_t ld, size_t es) {
  if (rows <= 0 || cols <= 0) return 0;
  return ((size_t)(rows - 1) * (size_t)ld + (size_t)cols) * es;
}

// a feature matrix: rows x cols, ld >= cols, 16-byte base and row pitch
saga_status check_mat(const void* ptr, int64_t rows, int64_t cols, int64_t ld, int64_t want_rows,
                      int64_t want_cols, size_t es, bool vec, const char* name) {
  if (rows != want_rows || cols != want_cols)
    return fail(SAGA_EINVAL, "%s: shape %lld x %lld, expected %lld x %lld", name, (long long)rows,
                (long long)cols, (long long)want_rows, (long long)want_cols);
  if (ld < cols) return fail(SAGA_EINVAL, "%s: ld %lld < cols %lld", name, (long long)ld, (long long)cols);
  if (rows > 0 && cols > 0 && !ptr) return fail(SAGA_EINVAL, "%s: null pointer", name);
  if (vec) {
    if ((uintptr_t)ptr % 16 != 0) return fail(SAGA_EINVAL, "%s: base not 16-byte aligned", name);
    if (((size_t)ld * es) % 16 != 0)
      return fail(SAGA_EINVAL, "%s: row pitch ld*elem = %zu not a multiple of 16", name, (size_t)ld * es);
  } else if ((uintptr_t)ptr % es != 0) {
    return fail(SAGA_EINVAL, "%s: misaligned base", name);
  }
  return SAGA_OK;
}

// Defaults sized to the graph: enough row blocks (about 2048) to fill the
// GPU on small graphs.  block_cost = the power of two at or below
// (E + row_cost * V) / 2048, clamped to [256, 4096]; seg_len = min(512,
// block_cost / 2).  The 2^21-vertex graph gets 4096 and 512.
int32_t default_block_cost(int64_t V, int64_t E, int32_t c) {
  const int64_t total = E + (int64_t)c * V;
  int64_t b = 256;
  while (b < 4096 && b * 2 <= total / 2048) b *= 2;
  return (int32_t)b;
}

saga_status resolve_opts(const saga_plan_opts* o, int64_t V, int64_t E, int32_t* T, int32_t* B,
                         int32_t* c) {
  const bool auto_t = !(o && o->seg_len), auto_b = !(o && o->block_cost);
  *c = o && o->row_cost ? o->row_cost : 4;
  *B = auto_b ? default_block_cost(V, E, *c) : o->block_cost;
  *T = auto_t ? (*B / 2 < 512 ? *B / 2 : 512) : o->seg_len;
  if (auto_b && *c > 0 && *T > 0)
    while (*B < *T + *c && *B < (1 << 30)) *B *= 2;
  if (*T <= 0 || *c <= 0) return fail(SAGA_EINVAL, "plan options: seg_len and row_cost must be > 0");
  if (*B < *T + *c) return fail(SAGA_EINVAL, "plan options: block_cost must be >= seg_len + row_cost");
  return SAGA_OK;
}

saga_status check_plan(const saga_plan* p) {
  if (!p) return fail(SAGA_EINVAL, "plan is null");
  if (!p->counts || !p->d_in || !p->perm || !p->seg_row || !p->block_ptr)
    return fail(SAGA_EINVAL, "plan is not built");
  return SAGA_OK;
}

saga_status check_rel(const saga_plan& p, const saga_rel_plan* r) {
  if (!r) return fail(SAGA_EINVAL, "rel plan is null");
  if (!r->counts || !r->rel_ptr || !r->pair_src || !r->edge_pair || !r->edge_norm)
    return fail(SAGA_EINVAL, "rel plan is not built");
  if (r->plan_counts != p.counts || r->num_edges != p.num_edges || r->num_src != p.num_src)
    return fail(SAGA_EINVAL, "rel plan was built on another plan");
  return SAGA_OK;
}

// bump allocator over a caller workspace
struct Carve {
  char* base;
  size_t cap, used = 0;
  Carve(void* b, size_t c) : base(static_cast<char*>(b)), cap(c) {}
  void* take(size_t n) {
    void* p = base ? base + used : nullptr;
    used = align256(used + n);
    return p;
  }
  bool fits() const { return used <= cap; }
};

saga::GatherArgs gather_args_from_plan(const saga_plan& p) {
  saga::GatherArgs a;
  memset(&a, 0, sizeof(a));
  a.block_cost = p.block_cost;
  a.row_ptr = p.row_ptr;
  a.col_idx = p.col_idx;
  a.d_in = p.d_in;
  a.d_out = p.d_out;
  a.perm = p.perm;
  a.row_seg_first = p.row_seg_first;
  a.seg_row = p.seg_row;
  a.seg_beg = p.seg_beg;
  a.seg_end = p.seg_end;
  a.block_ptr = p.block_ptr;
  a.counts = p.counts;
  a.max_blocks = p.max_blocks;
  a.max_split = p.max_split;
  return a;
}

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

saga_status gather_ws_bytes(const saga_plan& p, const saga_edge_op& op, int64_t feat,
                            size_t* bytes) {
  const size_t ps = saga::gather_partial_stride(op, feat);
  *bytes = align256((size_t)p.max_split_segments * ps * sizeof(float));
  return SAGA_OK;
}

saga_status validate_edge_op(const saga_plan& p, const saga_edge_op& op,
                             const saga_edge_inputs& in, const saga_mat& out) {
  const size_t es = esize(op.dtype);
  const int64_t F = in.src.cols;
  if (op.dtype != SAGA_F32 && op.dtype != SAGA_BF16) return fail(SAGA_EINVAL, "bad dtype");
  if (op.act < SAGA_ACT_NONE || op.act > SAGA_ACT_TANH) return fail(SAGA_EINVAL, "bad activation");
  if (F <= 0) return fail(SAGA_EINVAL, "src: no feature columns");
  // the split-row combine holds a row of at most 1024 columns
  if (F > 1024) return fail(SAGA_EUNSUPPORTED, "feature width %lld too large", (long long)F);
  int64_t src_rows = p.num_src;
  if (op.msg == SAGA_MSG_TYPED) {
    saga_status s0 = check_rel(p, in.rel);
    if (s0) return s0;
    if (op.reduce != SAGA_RED_SUM) return fail(SAGA_EUNSUPPORTED, "TYPED messages need SUM");
    src_rows = in.rel->max_pairs;
  }
  saga_status s = check_mat(in.src.ptr, in.src.rows, in.src.cols, in.src.ld, src_rows, F, es, true, "src");
  if (s) return s;
  int64_t out_cols = F;
  switch (op.msg) {
    case SAGA_MSG_COPY:
    case SAGA_MSG_SRC_NORM:
      if (op.reduce != SAGA_RED_SUM && op.reduce != SAGA_RED_MEAN && op.reduce != SAGA_RED_MAX)
        return fail(SAGA_EUNSUPPORTED, "COPY/SRC_NORM messages take SUM, MEAN or MAX");
      break;
    case SAGA_MSG_GAT: {
      if (op.reduce != SAGA_RED_SOFTMAX) return fail(SAGA_EUNSUPPORTED, "GAT messages need SOFTMAX");
      if (op.dtype != SAGA_F32) return fail(SAGA_EUNSUPPORTED, "GAT gather is float32 only");
      const int64_t H = op.heads;
      if (H <= 0 || F % H != 0 || (F / H) % 4 != 0 || F / 4 > 64)
        return fail(SAGA_EUNSUPPORTED, "GAT: heads must divide F into multiples of 4 (F <= 256)");
      if (op.head_mean && (!is_pow2(H) || !is_pow2(F / 4)))
        return fail(SAGA_EUNSUPPORTED, "GAT head mean needs power-of-two heads and F/4");
      s = check_mat(in.el.ptr, in.el.rows, in.el.cols, in.el.ld, p.num_src, H, 4, false, "el");
      if (s) return s;
      s = check_mat(in.er.ptr, in.er.rows, in.er.cols, in.er.ld, p.num_dst, H, 4, false, "er");
      if (s) return s;
      if (op.head_mean) out_cols = F / H;
      break;
    }
    case SAGA_MSG_GATED: {
      if (op.reduce != SAGA_RED_SUM) return fail(SAGA_EUNSUPPORTED, "GATED messages need SUM");
      if (op.dtype != SAGA_F32) return fail(SAGA_EUNSUPPORTED, "GATED gather is float32 only");
      if (F != 64) return fail(SAGA_EUNSUPPORTED, "GATED gather needs F == 64");
      const int64_t Fe = in.edge_feat.cols;
      if (Fe <= 0 || Fe > 16 || Fe % 4 != 0)
        return fail(SAGA_EUNSUPPORTED, "GATED: edge feature width must be 4, 8, 12 or 16");
      s = check_mat(in.gate_src.ptr, in.gate_src.rows, in.gate_src.cols, in.gate_src.ld, p.num_src, F, 4, true, "gate_src");
      if (s) return s;
      s = check_mat(in.gate_dst.ptr, in.gate_dst.rows, in.gate_dst.cols, in.gate_dst.ld, p.num_dst, F, 4, true, "gate_dst");
      if (s) return s;
      s = check_mat(in.edge_feat.ptr, in.edge_feat.rows, in.edge_feat.cols, in.edge_feat.ld, p.num_edges, Fe, 4, true, "edge_feat");
      if (s) return s;
      if (!in.w_edge) return fail(SAGA_EINVAL, "w_edge is null");
      break;
    }
    case SAGA_MSG_TYPED:
      break;  // src and rel are checked above
    default:
      return fail(SAGA_EINVAL, "bad message kind");
  }
  s = check_mat(out.ptr, out.rows, out.cols, out.ld, p.num_dst, out_cols, es, true, "out");
  if (s) return s;
  if (in.self.ptr) {
    if (op.msg != SAGA_MSG_COPY && op.msg != SAGA_MSG_SRC_NORM && op.msg != SAGA_MSG_TYPED)
      return fail(SAGA_EUNSUPPORTED, "self term: COPY, SRC_NORM or TYPED messages only");
    s = check_mat(in.self.ptr, in.self.rows, in.self.cols, in.self.ld, p.num_dst, out_cols, es,
                  false, "self");
    if (s) return s;
    if (range_overlap(out.ptr, mat_bytes(out.rows, out.cols, out.ld, es), in.self.ptr,
                      mat_bytes(in.self.rows, in.self.cols, in.self.ld, es)))
      return fail(SAGA_EINVAL, "output overlaps self");
  }
  const size_t ob = mat_bytes(out.rows, out.cols, out.ld, es);
  const void* ins[] = {in.src.ptr, in.el.ptr, in.er.ptr, in.gate_src.ptr, in.gate_dst.ptr,
                       in.edge_feat.ptr, p.row_ptr, p.col_idx};
  const size_t inb[] = {mat_bytes(in.src.rows, in.src.cols, in.src.ld, es),
                        mat_bytes(in.el.rows, in.el.cols, in.el.ld, 4),
                        mat_bytes(in.er.rows, in.er.cols, in.er.ld, 4),
                        mat_bytes(in.gate_src.rows, in.gate_src.cols, in.gate_src.ld, 4),
                        mat_bytes(in.gate_dst.rows, in.gate_dst.cols, in.gate_dst.ld, 4),
                        mat_bytes(in.edge_feat.rows, in.edge_feat.cols, in.edge_feat.ld, 4),
                        (size_t)(p.num_dst + 1) * 4, (size_t)p.num_edges * 4};
  for (int i = 0; i < 8; ++i)
    if (range_overlap(out.ptr, ob, ins[i], inb[i])) return fail(SAGA_EINVAL, "output overlaps an input");
  return SAGA_OK;
}

// GatherArgs of a validated call: plan, op, inputs, output, partials at ws
saga::GatherArgs fill_gather_args(const saga_plan& p, const saga_edge_op& op,
                                  const saga_edge_inputs& in, const saga_mat& out, void* ws) {
  saga::GatherArgs a = gather_args_from_plan(p);
  a.msg = op.msg;
  a.reduce = op.reduce;
  a.dtype = op.dtype;
  a.heads = op.msg == SAGA_MSG_GAT ? op.heads : 1;
  a.head_mean = op.msg == SAGA_MSG_GAT ? op.head_mean : 0;
  a.dst_norm = op.dst_norm;
  a.act = op.act;
  a.neg_slope = op.neg_slope;
  a.feat = (int)in.src.cols;
  a.out_cols = (int)out.cols;
  a.src = in.src.ptr;
  a.ld_src = in.src.ld;
  a.src_rows = in.src.rows;
  a.el = static_cast<const float*>(in.el.ptr);
  a.ld_el = in.el.ld;
  a.er = static_cast<const float*>(in.er.ptr);
  a.ld_er = in.er.ld;
  a.gsrc = static_cast<const float*>(in.gate_src.ptr);
  a.ld_gsrc = in.gate_src.ld;
  a.gdst = static_cast<const float*>(in.gate_dst.ptr);
  a.ld_gdst = in.gate_dst.ld;
  a.efeat = static_cast<const float*>(in.edge_feat.ptr);
  a.ld_efeat = in.edge_feat.ld;
  a.fe = (int)in.edge_feat.cols;
  a.w_edge = in.w_edge;
  a.gate_bias = in.gate_bias;
  a.bias = in.bias;
  a.self = in.self.ptr;
  a.ld_self = in.self.ld;
  if (op.msg == SAGA_MSG_TYPED) {
    a.col_idx = in.rel->edge_pair;
    a.edge_scale = in.rel->edge_norm;
    a.err2 = in.rel->counts + saga::kRelErr;
  }
  a.out = out.ptr;
  a.ld_out = out.ld;
  a.partial = static_cast<float*>(ws);
  a.pstride = (int64_t)saga::gather_partial_stride(op, in.src.cols);
  a.pcols = saga::gather_partial_cols(in.src.cols);
  return a;
}

saga_status run_gather(const saga_plan& p, const saga_edge_op& op, const saga_edge_inputs& in,
                       const saga_mat& out, void* ws, size_t ws_bytes, hipStream_t st) {
  saga_status s = validate_edge_op(p, op, in, out);
  if (s) return s;
  size_t need;
  gather_ws_bytes(p, op, in.src.cols, &need);
  if (p.max_split_segments > 0 && (!ws || ws_bytes < need))
    return fail(SAGA_EWORKSPACE, "gather workspace: need %zu bytes, got %zu", need, ws_bytes);
  if (p.num_dst == 0) return ok();
  const saga::GatherArgs a = fill_gather_args(p, op, in, out, ws);
  hipError_t e = saga::launch_gather(a, st);
  if (e != hipSuccess) return dev_fail(e, "gather launch");
  return ok();
}

// ---------------------------------------------------------------------------
// Gather with the next transform fused in (saga_scatter_apply_edge_gather_
// transform): workspace = the split-row partials, then the Gather output h
// (num_dst x F, the op's dtype; the earlier slices pass through it)
// ---------------------------------------------------------------------------
saga_status gather_xf_ws_bytes(const saga_plan& p, const saga_edge_op& op, int64_t feat,
                               size_t* part, size_t* total) {
  gather_ws_bytes(p, op, feat, part);
  // h, then W^T packed for the matrix cores (sized for 64 output columns)
  *total = *part + align256((size_t)p.num_dst * feat * esize(op.dtype)) +
           align256((size_t)saga::xf_pack_bytes(feat, (int)esize(op.dtype), 64));
  return SAGA_OK;
}

saga_status run_gather_transform(const saga_plan& p, const saga_edge_op& op,
                                 const saga_edge_inputs& in, const saga_next_transform& nx,
                                 const saga_mat& out, void* ws, size_t ws_bytes, hipStream_t st) {
  const size_t es = esize(op.dtype);
  const int64_t F = in.src.cols, N = nx.w.cols, V = p.num_dst;
  if (op.msg != SAGA_MSG_COPY || (op.reduce != SAGA_RED_SUM && op.reduce != SAGA_RED_MEAN))
    return fail(SAGA_EUNSUPPORTED, "gather + transform: COPY messages with SUM or MEAN only");
  if (F <= 0 || (F * (int64_t)es) % 128 != 0 || F * (int64_t)es > 4 * 128)
    return fail(SAGA_EUNSUPPORTED, "gather + transform: src must be 1 to 4 whole 128-byte lines "
                                   "wide (32..128 float32 or 64..256 bfloat16 columns)");
  if (in.src.rows * in.src.ld * (int64_t)es > (int64_t(1) << 32))
    return fail(SAGA_EUNSUPPORTED, "gather + transform: source matrix of 4 GiB or more");
  if (N < 1 || N > 64) return fail(SAGA_EUNSUPPORTED, "gather + transform: 1 to 64 output columns");
  saga_status s = check_mat(nx.w.ptr, nx.w.rows, nx.w.cols, nx.w.ld, F, N, es, false, "next.w");
  if (s) return s;
  if (nx.w.ld != N) return fail(SAGA_EINVAL, "next.w must be dense (ld == cols)");
  const int64_t epv = 16 / (int64_t)es;
  if (nx.split_col < 0 || (nx.split_col > 0 && (nx.split_col >= N || nx.split_col % epv != 0)))
    return fail(SAGA_EINVAL, "next.split_col must be 0, or in (0, N) and a multiple of %lld",
                (long long)epv);
  const int64_t head = nx.split_col > 0 ? nx.split_col : N;
  s = check_mat(out.ptr, out.rows, out.cols, out.ld, V, head, es, true, "out");
  if (s) return s;
  const saga_mat& t = nx.tail;
  if (nx.split_col > 0) {
    s = check_mat(t.ptr, t.rows, t.cols, t.ld, V, N - nx.split_col, es, true, "next.tail");
    if (s) return s;
  }
  size_t part, need;
  gather_xf_ws_bytes(p, op, F, &part, &need);
  if (!ws || ws_bytes < need)
    return fail(SAGA_EWORKSPACE, "gather + transform workspace: need %zu bytes, got %zu", need,
                ws_bytes);
  if ((uintptr_t)ws % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
  // h lives in the workspace; its shape is what the Gather's output check wants
  const saga_mat h = {static_cast<char*>(ws) + part, V, F, F};
  s = validate_edge_op(p, op, in, h);
  if (s) return s;
  const size_t ob = mat_bytes(out.rows, out.cols, out.ld, es);
  const size_t tb = nx.split_col > 0 ? mat_bytes(t.rows, t.cols, t.ld, es) : 0;
  const void* outs[2] = {out.ptr, nx.split_col > 0 ? t.ptr : nullptr};
  const size_t outb[2] = {ob, tb};
  const void* ins[5] = {in.src.ptr, nx.w.ptr, p.row_ptr, p.col_idx, ws};
  const size_t inb[5] = {mat_bytes(in.src.rows, in.src.cols, in.src.ld, es),
                         mat_bytes(nx.w.rows, nx.w.cols, nx.w.ld, es), (size_t)(V + 1) * 4,
                         (size_t)p.num_edges * 4, need};
  for (int i = 0; i < 2; ++i)
    for (int j = 0; j < 5; ++j)
      if (range_overlap(outs[i], outb[i], ins[j], inb[j]))
        return fail(SAGA_EINVAL, "gather + transform: an output overlaps an input or the workspace");
  if (nx.split_col > 0 && range_overlap(out.ptr, ob, t.ptr, tb))
    return fail(SAGA_EINVAL, "next.tail overlaps out");
  if (V == 0) return ok();
  saga::GatherArgs a = fill_gather_args(p, op, in, h, ws);
  a.xw = nx.w.ptr;
  a.xwt = reinterpret_cast<uint4*>(static_cast<char*>(ws) + part +
                                   align256((size_t)V * F * es));
  a.xn = (int)N;
  a.xsplit = nx.split_col;
  a.xout = out.ptr;
  a.ld_xout = out.ld;
  a.xtail = t.ptr;
  a.ld_xtail = t.ld;
  a.xrs = nx.row_scale_deg;
  hipError_t e = saga::launch_gather_transform(a, st);
  if (e != hipSuccess) return dev_fail(e, "gather + transform launch");
  return ok();
}

saga_status validate_gemm(const saga_gemm_op& op, const saga_cmat& a, const saga_cmat& w,
                          const saga_cmat& a2, const saga_cmat& w2, const saga_mat& out) {
  if (op.dtype != SAGA_F32 && op.dtype != SAGA_BF16) return fail(SAGA_EINVAL, "bad dtype");
  if (op.mode < SAGA_GEMM_PLAIN || op.mode > SAGA_GEMM_GRU) return fail(SAGA_EINVAL, "bad mode");
  if (op.act < SAGA_ACT_NONE || op.act > SAGA_ACT_TANH) return fail(SAGA_EINVAL, "bad activation");
  const size_t es = esize(op.dtype);
  const int64_t M = a.rows, K = a.cols, N = w.cols;
  if (M < 0 || K <= 0 || N <= 0) return fail(SAGA_EINVAL, "gemm: empty operand");
  saga_status s = check_mat(a.ptr, a.rows, a.cols, a.ld, M, K, es, true, "a");
  if (s) return s;
  s = check_mat(w.ptr, w.rows, w.cols, w.ld, K, N, es, false, "w");
  if (s) return s;
  if (op.mode != SAGA_GEMM_PLAIN) {
    s = check_mat(a2.ptr, a2.rows, a2.cols, a2.ld, M, a2.cols, es, true, "a2");
    if (s) return s;
    if (a2.cols <= 0) return fail(SAGA_EINVAL, "a2: no columns");
    s = check_mat(w2.ptr, w2.rows, w2.cols, w2.ld, a2.cols, N, es, false, "w2");
    if (s) return s;
  }
  int64_t out_cols = N;
  if (op.mode == SAGA_GEMM_GRU) {
    if (N % 3 != 0) return fail(SAGA_EINVAL, "GRU: w must have 3F columns");
    out_cols = N / 3;
    if (out_cols != 16 && out_cols != 32 && out_cols != 48 && out_cols != 64)
      return fail(SAGA_EUNSUPPORTED, "GRU: F must be 16, 32, 48 or 64");
    if (a2.cols != out_cols) return fail(SAGA_EINVAL, "GRU: hidden state a2 must have F columns");
  } else if (N > 4096) {
    return fail(SAGA_EUNSUPPORTED, "gemm: N too large");
  }
  if (op.split_col < 0 || (op.split_col > 0 && (op.mode == SAGA_GEMM_GRU || op.split_col >= out_cols)))
    return fail(SAGA_EINVAL, "split_col must be 0, or in (0, N) for PLAIN / CONCAT");
  const int64_t head = op.split_col > 0 ? op.split_col : out_cols;
  s = check_mat(out.ptr, out.rows, out.cols, out.ld, M, head, es, false, "out");
  if (s) return s;
  const size_t ob = mat_bytes(out.rows, out.cols, out.ld, es);
  const saga_mat& t = op.tail;
  const size_t tb = op.split_col > 0 ? mat_bytes(t.rows, t.cols, t.ld, es) : 0;
  if (op.split_col > 0) {
    s = check_mat(t.ptr, t.rows, t.cols, t.ld, M, out_cols - op.split_col, es, false, "tail");
    if (s) return s;
    if (range_overlap(out.ptr, ob, t.ptr, tb)) return fail(SAGA_EINVAL, "tail overlaps out");
  }
  const void* outs[2] = {out.ptr, op.split_col > 0 ? t.ptr : nullptr};
  const size_t outb[2] = {ob, tb};
  for (int i = 0; i < 2; ++i)
    if (range_overlap(outs[i], outb[i], a.ptr, mat_bytes(a.rows, a.cols, a.ld, es)) ||
        range_overlap(outs[i], outb[i], w.ptr, mat_bytes(w.rows, w.cols, w.ld, es)) ||
        range_overlap(outs[i], outb[i], a2.ptr, mat_bytes(a2.rows, a2.cols, a2.ld, es)) ||
        range_overlap(outs[i], outb[i], w2.ptr, mat_bytes(w2.rows, w2.cols, w2.ld, es)))
      return fail(SAGA_EINVAL, "output overlaps an input");
  return SAGA_OK;
}

size_t gemm_ws_bytes(const saga_gemm_op& op, int64_t k, int64_t k2, int64_t n) {
  return saga::gemm_workspace_bytes(op.dtype, op.mode, n, k, op.mode == SAGA_GEMM_PLAIN ? 0 : k2);
}

saga_status run_gemm(const saga_gemm_op& op, const saga_cmat& a, const saga_cmat& w,
                     const saga_cmat& a2, const saga_cmat& w2, const float* bias,
                     const float* bias2, const saga_mat& out, void* ws, size_t ws_bytes,
                     hipStream_t st) {
  saga_status s = validate_gemm(op, a, w, a2, w2, out);
  if (s) return s;
  const size_t need = gemm_ws_bytes(op, a.cols, a2.cols, w.cols);
  if (!ws || ws_bytes < need)
    return fail(SAGA_EWORKSPACE, "apply_vertex workspace: need %zu bytes, got %zu", need, ws_bytes);
  if ((uintptr_t)ws % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
  {
    const size_t es = esize(op.dtype);
    if (range_overlap(ws, need, out.ptr, mat_bytes(out.rows, out.cols, out.ld, es)) ||
        (op.split_col > 0 &&
         range_overlap(ws, need, op.tail.ptr, mat_bytes(op.tail.rows, op.tail.cols, op.tail.ld, es))) ||
        range_overlap(ws, need, a.ptr, mat_bytes(a.rows, a.cols, a.ld, es)) ||
        range_overlap(ws, need, w.ptr, mat_bytes(w.rows, w.cols, w.ld, es)) ||
        range_overlap(ws, need, a2.ptr, mat_bytes(a2.rows, a2.cols, a2.ld, es)) ||
        range_overlap(ws, need, w2.ptr, mat_bytes(w2.rows, w2.cols, w2.ld, es)))
      return fail(SAGA_EINVAL, "workspace overlaps an argument");
  }
  saga::GemmArgs g;
  memset(&g, 0, sizeof(g));
  g.dtype = op.dtype;
  g.mode = op.mode;
  g.act = op.act;
  g.M = a.rows;
  g.N = w.cols;
  g.K = a.cols;
  g.K2 = a2.cols;
  g.a = a.ptr;
  g.lda = a.ld;
  g.w = w.ptr;
  g.ldw = w.ld;
  g.a2 = a2.ptr;
  g.lda2 = a2.ld;
  g.w2 = w2.ptr;
  g.ldw2 = w2.ld;
  g.bias = bias;
  g.bias2 = bias2;
  g.row_scale_deg = op.row_scale_deg;
  g.out = out.ptr;
  g.ldo = out.ld;
  if (op.split_col > 0) {
    g.split = op.split_col;
    g.out2 = op.tail.ptr;
    g.ldo2 = op.tail.ld;
  }
  g.ws = ws;
  g.ws_bytes = ws_bytes;
  hipError_t e = saga::launch_gemm(g, st);
  if (e != hipSuccess) return dev_fail(e, "gemm launch");
  return ok();
}

// -------------------------------------------------------------------------
// layers
// -------------------------------------------------------------------------
struct LayerPlanWs {
  size_t bytes;
};

// Leading dimension of a layer intermediate that the gather reads by rows:
// rows of up to 128 bytes are padded to a power of two (never straddling a
// 128-byte L2 line), longer rows to a multiple of 64 bytes (each row then
// touches a whole number of lines).
int64_t ld_for(int64_t cols, int32_t t) {
  const int64_t es = t == SAGA_BF16 ? 2 : 4;
  int64_t bytes = cols * es;
  if (bytes <= 128) {
    int64_t p = 16;
    while (p < bytes) p <<= 1;
    bytes = p;
  } else {
    bytes = round_up(bytes, 64);
  }
  return bytes / es;
}

// ---------------------------------------------------------------------------
// unfused baseline: index-select into an E x ldm edge tensor, then reduce
// ---------------------------------------------------------------------------
size_t unfused_msg_bytes(const saga_plan& p, const saga_edge_op& op, int64_t feat, int64_t* ldm) {
  const int32_t t = op.dtype == SAGA_BF16 ? SAGA_BF16 : SAGA_F32;
  *ldm = ld_for(feat, t);
  return align256((size_t)p.num_edges * (size_t)*ldm * esize(t));
}

saga_status unfused_ws_bytes(const saga_plan& p, const saga_edge_op& op, int64_t feat,
                             size_t* bytes) {
  int64_t ldm;
  size_t pb;
  gather_ws_bytes(p, op, feat, &pb);
  *bytes = unfused_msg_bytes(p, op, feat, &ldm) + pb;
  return SAGA_OK;
}

saga_status run_gather_unfused(const saga_plan& p, const saga_edge_op& op,
                               const saga_edge_inputs& in, const saga_mat& out, void* ws,
                               size_t ws_bytes, hipStream_t st) {
  if (op.msg != SAGA_MSG_COPY && op.msg != SAGA_MSG_SRC_NORM)
    return fail(SAGA_EUNSUPPORTED, "unfused path: msg must be COPY or SRC_NORM");
  if (op.reduce != SAGA_RED_SUM && op.reduce != SAGA_RED_MEAN && op.reduce != SAGA_RED_MAX)
    return fail(SAGA_EUNSUPPORTED, "unfused path: reduce must be SUM, MEAN or MAX");
  saga_status s = validate_edge_op(p, op, in, out);
  if (s) return s;
  int64_t ldm;
  const size_t mb = unfused_msg_bytes(p, op, in.src.cols, &ldm);
  size_t need;
  unfused_ws_bytes(p, op, in.src.cols, &need);
  if (!ws || ws_bytes < need)
    return fail(SAGA_EWORKSPACE, "unfused workspace: need %zu bytes, got %zu", need, ws_bytes);
  if ((uintptr_t)ws % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
  const size_t es = esize(op.dtype);
  if (range_overlap(ws, need, out.ptr, mat_bytes(out.rows, out.cols, out.ld, es)) ||
      range_overlap(ws, need, in.src.ptr, mat_bytes(in.src.rows, in.src.cols, in.src.ld, es)))
    return fail(SAGA_EINVAL, "workspace overlaps an argument");
  if (p.num_dst == 0) return ok();
  saga::GatherArgs a = gather_args_from_plan(p);
  a.msg = op.msg;
  a.reduce = op.reduce;
  a.dtype = op.dtype;
  a.heads = 1;
  a.dst_norm = op.dst_norm;
  a.act = op.act;
  a.feat = (int)in.src.cols;
  a.out_cols = (int)out.cols;
  a.src = in.src.ptr;
  a.ld_src = in.src.ld;
  a.bias = in.bias;
  a.out = out.ptr;
  a.ld_out = out.ld;
  char* w = static_cast<char*>(ws);
  a.partial = reinterpret_cast<float*>(w + mb);
  a.pstride = (int64_t)saga::gather_partial_stride(op, in.src.cols);
  a.pcols = saga::gather_partial_cols(in.src.cols);
  hipError_t e = saga::launch_unfused(a, p.num_edges, w, ldm, st);
  if (e != hipSuccess) return dev_fail(e, "unfused gather launch");
  return ok();
}

// ---------------------------------------------------------------------------
// LSTM Gather
// ---------------------------------------------------------------------------
constexpr size_t kLstmWs = 256;

saga_status run_lstm(const saga_plan& p, const saga_cmat& gx, const saga_cmat& whh,
                     const saga_mat& out, void* ws, size_t ws_bytes, hipStream_t st,
                     int64_t perm_begin = 0, int64_t perm_end = -1) {
  if (perm_end < 0) perm_end = p.num_dst;
  if (perm_begin < 0 || perm_begin > perm_end || perm_end > p.num_dst)
    return fail(SAGA_EINVAL, "lstm gather: perm range [%lld, %lld) outside [0, %d]",
                (long long)perm_begin, (long long)perm_end, p.num_dst);
  const int64_t H = whh.rows;
  if (H != 32 && H != 64 && H != 128)
    return fail(SAGA_EUNSUPPORTED, "lstm gather: hidden size must be 32, 64 or 128 (got %lld)",
                (long long)H);
  saga_status s = check_mat(gx.ptr, gx.rows, gx.cols, gx.ld, p.num_src, 4 * H, 4, true, "gates_x");
  if (s) return s;
  s = check_mat(whh.ptr, whh.rows, whh.cols, whh.ld, H, 4 * H, 4, false, "w_hh");
  if (s) return s;
  s = check_mat(out.ptr, out.rows, out.cols, out.ld, p.num_dst, H, 4, false, "out");
  if (s) return s;
  if (!ws || ws_bytes < kLstmWs)
    return fail(SAGA_EWORKSPACE, "lstm workspace: need %zu bytes, got %zu", kLstmWs, ws_bytes);
  if ((uintptr_t)ws % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
  const size_t ob = mat_bytes(out.rows, out.cols, out.ld, 4);
  if (range_overlap(out.ptr, ob, gx.ptr, mat_bytes(gx.rows, gx.cols, gx.ld, 4)) ||
      range_overlap(out.ptr, ob, whh.ptr, mat_bytes(whh.rows, whh.cols, whh.ld, 4)) ||
      range_overlap(out.ptr, ob, ws, kLstmWs))
    return fail(SAGA_EINVAL, "output overlaps an input or the workspace");
  saga::LstmArgs a;
  memset(&a, 0, sizeof(a));
  a.row_ptr = p.row_ptr;
  a.col_idx = p.col_idx;
  a.perm = p.perm;
  a.counts = p.counts;
  a.num_dst = p.num_dst;
  a.hidden = (int)H;
  a.gates_x = static_cast<const float*>(gx.ptr);
  a.ld_gx = gx.ld;
  a.w_hh = static_cast<const float*>(whh.ptr);
  a.ld_whh = whh.ld;
  a.out = static_cast<float*>(out.ptr);
  a.ld_out = out.ld;
  a.queue = static_cast<int32_t*>(ws);
  a.perm_begin = (int32_t)perm_begin;
  a.perm_end = (int32_t)perm_end;
  hipError_t e = saga::launch_lstm_gather(a, st);
  if (e != hipSuccess) return dev_fail(e, "lstm gather launch");
  return ok();
}

// ---------------------------------------------------------------------------
// R-GCN: per-relation transform of the distinct (relation, source) pairs
// ---------------------------------------------------------------------------
saga_status run_rel_transform(const saga_rel_plan& r, int32_t dtype, const saga_cmat& x,
                              const saga_cmat& w, const saga_mat& out, void* ws, size_t ws_bytes,
                              hipStream_t st) {
  if (dtype != SAGA_F32 && dtype != SAGA_BF16) return fail(SAGA_EINVAL, "bad dtype");
  const size_t es = esize(dtype);
  const int64_t K = x.cols, N = w.cols, R = r.num_rel;
  if (K <= 0 || N <= 0) return fail(SAGA_EINVAL, "rel transform: empty operand");
  if (N > 4096) return fail(SAGA_EUNSUPPORTED, "rel transform: N too large");
  saga_status s = check_mat(x.ptr, x.rows, x.cols, x.ld, r.num_src, K, es, true, "x");
  if (s) return s;
  s = check_mat(w.ptr, w.rows, w.cols, w.ld, R * K, N, es, false, "w");
  if (s) return s;
  s = check_mat(out.ptr, out.rows, out.cols, out.ld, r.max_pairs, N, es, false, "out");
  if (s) return s;
  const size_t need = saga::gemm_grouped_workspace_bytes(dtype, (int)R, N, K);
  if (!ws || ws_bytes < need)
    return fail(SAGA_EWORKSPACE, "rel transform workspace: need %zu bytes, got %zu", need, ws_bytes);
  if ((uintptr_t)ws % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
  const size_t ob = mat_bytes(out.rows, out.cols, out.ld, es);
  const size_t xb = mat_bytes(x.rows, x.cols, x.ld, es), wb = mat_bytes(w.rows, w.cols, w.ld, es);
  if (range_overlap(out.ptr, ob, x.ptr, xb) || range_overlap(out.ptr, ob, w.ptr, wb) ||
      range_overlap(out.ptr, ob, ws, need))
    return fail(SAGA_EINVAL, "output overlaps an input or the workspace");
  if (range_overlap(ws, need, x.ptr, xb) || range_overlap(ws, need, w.ptr, wb))
    return fail(SAGA_EINVAL, "workspace overlaps an argument");
  if (r.max_pairs == 0) return ok();
  saga::GemmArgs g;
  memset(&g, 0, sizeof(g));
  g.dtype = dtype;
  g.mode = SAGA_GEMM_PLAIN;
  g.M = r.max_pairs;
  g.N = N;
  g.K = K;
  g.a = x.ptr;
  g.lda = x.ld;
  g.w = w.ptr;
  g.ldw = w.ld;
  g.out = out.ptr;
  g.ldo = out.ld;
  g.ws = ws;
  g.ws_bytes = ws_bytes;
  g.arow = r.pair_src;
  g.grp_ptr = r.rel_ptr;
  g.groups = (int)R;
  g.err1 = r.plan_counts + saga::kErrFlags;
  g.err2 = r.counts + saga::kRelErr;
  hipError_t e = saga::launch_gemm_grouped(g, st);
  if (e != hipSuccess) return dev_fail(e, "rel transform launch");
  return ok();
}

saga_status layer_check_desc(const saga_plan& p, const saga_layer_desc& d) {
  if (p.num_dst != p.num_src) return fail(SAGA_EINVAL, "layers need num_src == num_dst");
  if (d.in_feat <= 0 || d.out_feat <= 0) return fail(SAGA_EINVAL, "layer feature sizes must be > 0");
  if (d.dtype != SAGA_F32 && d.dtype != SAGA_BF16) return fail(SAGA_EINVAL, "bad dtype");
  switch (d.kind) {
    case SAGA_LAYER_GCN:
      if (!d.w) return fail(SAGA_EINVAL, "GCN: w is null");
      break;
    case SAGA_LAYER_GAT:
      if (d.dtype != SAGA_F32) return fail(SAGA_EUNSUPPORTED, "GAT layer is float32 only");
      if (!d.w || !d.attn_l || !d.attn_r) return fail(SAGA_EINVAL, "GAT: null weights");
      if (d.heads <= 0) return fail(SAGA_EINVAL, "GAT: heads must be > 0");
      break;
    case SAGA_LAYER_SAGE_POOL:
      if (d.dtype != SAGA_F32) return fail(SAGA_EUNSUPPORTED, "SAGE layer is float32 only");
      if (!d.w || !d.w_pool) return fail(SAGA_EINVAL, "SAGE: null weights");
      break;
    case SAGA_LAYER_SAGE_LSTM:
      if (d.dtype != SAGA_F32) return fail(SAGA_EUNSUPPORTED, "SAGE-LSTM layer is float32 only");
      if (!d.w || !d.w_ih || !d.w_hh) return fail(SAGA_EINVAL, "SAGE-LSTM: null weights");
      if (d.hidden != 32 && d.hidden != 64 && d.hidden != 128)
        return fail(SAGA_EUNSUPPORTED, "SAGE-LSTM: hidden must be 32, 64 or 128");
      break;
    case SAGA_LAYER_RGCN: {
      if (!d.w || !d.w_self) return fail(SAGA_EINVAL, "RGCN: null weights");
      saga_status s = check_rel(p, d.rel);
      if (s) return s;
      break;
    }
    case SAGA_LAYER_GATED_GRU:
      if (d.dtype != SAGA_F32) return fail(SAGA_EUNSUPPORTED, "gated layer is float32 only");
      if (!d.w_e || !d.w_ih || !d.w_hh) return fail(SAGA_EINVAL, "gated: null weights");
      if (d.in_feat != d.out_feat) return fail(SAGA_EINVAL, "gated: in_feat must equal out_feat");
      break;
    default:
      return fail(SAGA_EINVAL, "bad layer kind");
  }
  return SAGA_OK;
}

// returns workspace bytes; with a non-null base, also carves the buffers
struct LayerBufs {
  void* z = nullptr; int64_t ldz = 0;      // GCN Z / GAT [z|el|er] / SAGE P / gated S_src
  void* z2 = nullptr; int64_t ldz2 = 0;    // SAGE A / gated S_dst / GCN agg (aggregate-first)
  void* z3 = nullptr; int64_t ldz3 = 0;    // gated a
  float* wext = nullptr; int64_t ldw = 0;  // GAT folded weights
  void* part = nullptr;
  size_t part_bytes = 0;
  void* gws = nullptr;                     // packed weights of the layer's GEMMs
  size_t gws_bytes = 0;
  void* lstm_q = nullptr;                  // LSTM Gather work-queue counter
};

bool gcn_transform_first(const saga_layer_desc& d) { return d.out_feat <= d.in_feat; }

// Columns of a gathered row that fill whole 128-byte L2 lines, when the row
// is longer than one line but not a whole number of lines (0 otherwise):
// the transform then writes those columns and the rest as two matrices, and
// each is gathered by its own call, so no gathered row straddles a line
// shared with its neighbour (F = 41 float32: 32 + 9 columns instead of one
// 192-byte row over two lines).
int64_t line_split(int64_t cols, int32_t t) {
  const int64_t es = t == SAGA_BF16 ? 2 : 4, per_line = 128 / es;
  if (cols <= per_line || cols % per_line == 0) return 0;
  return cols / per_line * per_line;
}

size_t layer_carve(const saga_plan& p, const saga_layer_desc& d, void* base, LayerBufs* b) {
  Carve c(base, (size_t)-1);
  const int64_t V = p.num_dst;
  const int32_t t = d.dtype;
  const size_t es = esize(t);
  saga_edge_op op;
  memset(&op, 0, sizeof(op));
  int64_t gfeat = d.out_feat;
  switch (d.kind) {
    case SAGA_LAYER_GCN:
      if (gcn_transform_first(d)) {
        const int64_t sp = line_split(d.out_feat, t);
        b->ldz = ld_for(sp > 0 ? sp : d.out_feat, t);
        b->z = c.take((size_t)V * b->ldz * es);
        if (sp > 0) {  // the columns past the last whole line
          b->ldz3 = ld_for(d.out_feat - sp, t);
          b->z3 = c.take((size_t)V * b->ldz3 * es);
        }
        gfeat = d.out_feat;
      } else {
        b->ldz2 = ld_for(d.in_feat, t);
        b->z2 = c.take((size_t)V * b->ldz2 * es);
        gfeat = d.in_feat;
      }
      op.reduce = SAGA_RED_SUM;
      break;
    case SAGA_LAYER_GAT: {
      const int64_t F = d.head_mean ? (int64_t)d.out_feat * d.heads : d.out_feat;
      const int64_t cols = F + 2 * d.heads;
      b->ldw = ld_for(cols, SAGA_F32);
      b->wext = static_cast<float*>(c.take((size_t)d.in_feat * b->ldw * 4));
      b->ldz = ld_for(cols, SAGA_F32);
      b->z = c.take((size_t)V * b->ldz * 4);
      op.reduce = SAGA_RED_SOFTMAX;
      op.heads = d.heads;
      gfeat = F;
      break;
    }
    case SAGA_LAYER_SAGE_POOL:
      b->ldz = ld_for(d.in_feat, t);
      b->z = c.take((size_t)V * b->ldz * es);
      b->ldz2 = ld_for(d.in_feat, t);
      b->z2 = c.take((size_t)V * b->ldz2 * es);
      op.reduce = SAGA_RED_MAX;
      gfeat = d.in_feat;
      break;
    case SAGA_LAYER_SAGE_LSTM:
      b->ldz = 4 * (int64_t)d.hidden;  // P rows of 512 B (H = 32) to 2 KB, whole lines
      b->z = c.take((size_t)V * b->ldz * 4);
      b->ldz2 = ld_for(d.hidden, SAGA_F32);
      b->z2 = c.take((size_t)V * b->ldz2 * 4);
      b->lstm_q = c.take(kLstmWs);
      op.reduce = SAGA_RED_SUM;
      gfeat = 0;
      break;
    case SAGA_LAYER_RGCN:
      // T: the pair rows (rel transform); S = X W_self + b (the self term)
      b->ldz = ld_for(d.out_feat, t);
      b->z = c.take((size_t)d.rel->max_pairs * b->ldz * es);
      b->ldz2 = ld_for(d.out_feat, t);
      b->z2 = c.take((size_t)V * b->ldz2 * es);
      op.reduce = SAGA_RED_SUM;
      gfeat = d.out_feat;
      break;
    case SAGA_LAYER_GATED_GRU:
      b->ldz = ld_for(d.in_feat, t);
      b->z = c.take((size_t)V * b->ldz * es);
      b->ldz2 = b->ldz;
      b->z2 = c.take((size_t)V * b->ldz2 * es);
      b->ldz3 = b->ldz;
      b->z3 = c.take((size_t)V * b->ldz3 * es);
      op.reduce = SAGA_RED_SUM;
      gfeat = d.in_feat;
      break;
  }
  size_t pb = 0;
  if (gfeat > 0) gather_ws_bytes(p, op, gfeat, &pb);
  b->part_bytes = pb;
  b->part = c.take(pb);
  // one region for the packed weights, sized for the largest GEMM of the layer
  saga_gemm_op g;
  memset(&g, 0, sizeof(g));
  g.dtype = t;
  g.mode = SAGA_GEMM_PLAIN;
  const int64_t Fi = d.in_feat, Fo = d.out_feat;
  size_t gb = 0;
  switch (d.kind) {
    case SAGA_LAYER_GCN:
      gb = gemm_ws_bytes(g, Fi, 0, Fo);
      break;
    case SAGA_LAYER_GAT: {
      const int64_t F = d.head_mean ? Fo * d.heads : Fo;
      gb = gemm_ws_bytes(g, Fi, 0, F + 2 * d.heads);
      break;
    }
    case SAGA_LAYER_SAGE_POOL: {
      gb = gemm_ws_bytes(g, Fi, 0, Fi);
      g.mode = SAGA_GEMM_CONCAT;
      gb = std::max(gb, gemm_ws_bytes(g, Fi, Fi, Fo));
      break;
    }
    case SAGA_LAYER_GATED_GRU: {
      gb = gemm_ws_bytes(g, Fi, 0, Fi);
      g.mode = SAGA_GEMM_GRU;
      gb = std::max(gb, gemm_ws_bytes(g, Fi, Fi, 3 * Fi));
      break;
    }
    case SAGA_LAYER_SAGE_LSTM: {
      gb = gemm_ws_bytes(g, Fi, 0, 4 * (int64_t)d.hidden);
      g.mode = SAGA_GEMM_CONCAT;
      gb = std::max(gb, gemm_ws_bytes(g, Fi, d.hidden, Fo));
      break;
    }
    case SAGA_LAYER_RGCN:
      gb = std::max(gemm_ws_bytes(g, Fi, 0, Fo),
                    saga::gemm_grouped_workspace_bytes(t, d.rel->num_rel, Fo, Fi));
      break;
  }
  b->gws_bytes = gb;
  b->gws = c.take(gb);
  return c.used;
}

// ---------------------------------------------------------------------------
// Stage tracing (saga_trace_stages): after each stage of saga_layer, record
// the next of the caller's events on the layer's stream and, with markers,
// launch k_stage_mark, an empty kernel that delimits the stages in a
// counter profile's dispatch list (k_stage_begin opens each traced layer
// call).  With markers, the host side of the call is also bracketed by
// roctx ranges ("saga_layer", and "saga stage k" around the enqueue of
// stage k) for a timeline trace (rocprofv3 --marker-trace).
// Thread-local; off unless set.
// ---------------------------------------------------------------------------
__global__ void k_stage_begin() {}
__global__ void k_stage_mark() {}

thread_local std::vector<hipEvent_t> g_stage_events;
thread_local int g_stage_next = 0;
thread_local int g_stage_markers = 0;
thread_local int g_range_depth = 0;  // roctx ranges this layer call has open

void stage_range_push(int k) {
  char name[32];
  snprintf(name, sizeof(name), "saga stage %d", k);
  roctxRangePushA(name);
  ++g_range_depth;
}

void stage_ranges_close() {
  for (; g_range_depth > 0; --g_range_depth) roctxRangePop();
}

// after stage k: record event k, mark the dispatch list, and (last ==
// false) open stage k + 1's range
saga_status stage_done(hipStream_t st, bool last = false) {
  if (g_stage_next < (int)g_stage_events.size()) {
    const hipError_t e = hipEventRecord(g_stage_events[g_stage_next], st);
    if (e != hipSuccess) return dev_fail(e, "stage event");
  }
  ++g_stage_next;
  if (g_stage_markers) {
    hipLaunchKernelGGL(k_stage_mark, dim3(1), dim3(64), 0, st);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return dev_fail(e, "stage marker");
    if (g_range_depth > 1) {  // this stage's range
      roctxRangePop();
      --g_range_depth;
    }
    if (!last) stage_range_push(g_stage_next);
  }
  return SAGA_OK;
}

saga_status run_layer(const saga_plan& p, const saga_layer_desc& d, const saga_cmat& x,
                      const saga_cmat& ef, const saga_mat& out, void* ws, size_t ws_bytes,
                      hipStream_t st) {
  saga_status s = layer_check_desc(p, d);
  if (s) return s;
  LayerBufs b;
  const size_t need = layer_carve(p, d, nullptr, &b);
  if (!ws || ws_bytes < need)
    return fail(SAGA_EWORKSPACE, "layer workspace: need %zu bytes, got %zu", need, ws_bytes);
  if ((uintptr_t)ws % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
  b = LayerBufs();
  layer_carve(p, d, ws, &b);
  g_stage_next = 0;
  if (g_stage_markers) {
    roctxRangePushA("saga_layer");
    ++g_range_depth;
    stage_range_push(0);
    hipLaunchKernelGGL(k_stage_begin, dim3(1), dim3(64), 0, st);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return dev_fail(e, "stage marker");
  }
  const size_t es = esize(d.dtype);
  const int64_t V = p.num_dst, Fi = d.in_feat, Fo = d.out_feat;
  s = check_mat(x.ptr, x.rows, x.cols, x.ld, V, Fi, es, true, "x");
  if (s) return s;
  const void* wsend = static_cast<char*>(ws) + need;
  if (range_overlap(out.ptr, mat_bytes(out.rows, out.cols, out.ld, es), ws,
                    (size_t)((char*)wsend - (char*)ws)))
    return fail(SAGA_EINVAL, "output overlaps the workspace");

  saga_gemm_op g;
  memset(&g, 0, sizeof(g));
  g.dtype = d.dtype;
  saga_edge_op op;
  memset(&op, 0, sizeof(op));
  op.dtype = d.dtype;
  saga_edge_inputs in;
  memset(&in, 0, sizeof(in));
  const saga_cmat none = {nullptr, 0, 0, 0};

  switch (d.kind) {
    case SAGA_LAYER_GCN: {
      if (gcn_transform_first(d)) {
        // Z = d_out^-1/2 (X W); out = act(d_in^-1/2 sum_u Z_u + b)
        const int64_t sp = line_split(Fo, d.dtype);
        g.mode = SAGA_GEMM_PLAIN;
        g.row_scale_deg = p.d_out;
        if (sp > 0) {
          g.split_col = (int32_t)sp;
          g.tail = saga_mat{b.z3, V, Fo - sp, b.ldz3};
        }
        s = run_gemm(g, x, saga_cmat{d.w, Fi, Fo, Fo}, none, none, nullptr, nullptr,
                     saga_mat{b.z, V, sp > 0 ? sp : Fo, b.ldz}, b.gws, b.gws_bytes, st);
        if (s) return s;
        if ((s = stage_done(st))) return s;
        op.msg = SAGA_MSG_COPY;
        op.reduce = SAGA_RED_SUM;
        op.dst_norm = 1;
        op.act = d.act;
        if (sp == 0) {
          in.src = saga_cmat{b.z, V, Fo, b.ldz};
          in.bias = d.b;
          s = run_gather(p, op, in, out, b.part, b.part_bytes, st);
          if (s) return s;
          return stage_done(st, true);
        }
        // the whole-line columns, then the rest, into the two column ranges of out
        in.src = saga_cmat{b.z, V, sp, b.ldz};
        in.bias = d.b;
        s = run_gather(p, op, in, saga_mat{out.ptr, out.rows, sp, out.ld}, b.part, b.part_bytes, st);
        if (s) return s;
        if ((s = stage_done(st))) return s;
        in.src = saga_cmat{b.z3, V, Fo - sp, b.ldz3};
        in.bias = d.b ? d.b + sp : nullptr;
        s = run_gather(p, op, in,
                       saga_mat{static_cast<char*>(out.ptr) + sp * es, out.rows, Fo - sp, out.ld},
                       b.part, b.part_bytes, st);
        if (s) return s;
        return stage_done(st, true);
      }
      // aggregate first: agg = d_in^-1/2 sum_u d_out(u)^-1/2 X_u; out = act(agg W + b)
      op.msg = SAGA_MSG_SRC_NORM;
      op.reduce = SAGA_RED_SUM;
      op.dst_norm = 1;
      in.src = x;
      s = run_gather(p, op, in, saga_mat{b.z2, V, Fi, b.ldz2}, b.part, b.part_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      g.mode = SAGA_GEMM_PLAIN;
      g.act = d.act;
      s = run_gemm(g, saga_cmat{b.z2, V, Fi, b.ldz2}, saga_cmat{d.w, Fi, Fo, Fo}, none, none,
                   d.b, nullptr, out, b.gws, b.gws_bytes, st);
      if (s) return s;
      return stage_done(st, true);
    }
    case SAGA_LAYER_GAT: {
      const int64_t H = d.heads;
      const int64_t F = d.head_mean ? Fo * H : Fo;
      const int64_t cols = F + 2 * H;
      hipError_t e = saga::launch_fold_attention(static_cast<const float*>(d.w), Fi, F, (int)H,
                                                 d.attn_l, d.attn_r, b.wext, b.ldw, st);
      if (e != hipSuccess) return dev_fail(e, "fold launch");
      g.mode = SAGA_GEMM_PLAIN;
      s = run_gemm(g, x, saga_cmat{b.wext, Fi, cols, b.ldw}, none, none, nullptr, nullptr,
                   saga_mat{b.z, V, cols, b.ldz}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      const float* z = static_cast<const float*>(b.z);
      op.msg = SAGA_MSG_GAT;
      op.reduce = SAGA_RED_SOFTMAX;
      op.heads = (int32_t)H;
      op.head_mean = d.head_mean;
      op.neg_slope = d.neg_slope;
      op.act = d.act;
      in.src = saga_cmat{z, V, F, b.ldz};
      in.el = saga_cmat{z + F, V, H, b.ldz};
      in.er = saga_cmat{z + F + H, V, H, b.ldz};
      in.bias = d.b;
      s = run_gather(p, op, in, out, b.part, b.part_bytes, st);
      if (s) return s;
      return stage_done(st, true);
    }
    case SAGA_LAYER_SAGE_POOL: {
      g.mode = SAGA_GEMM_PLAIN;
      g.act = SAGA_ACT_RELU;
      s = run_gemm(g, x, saga_cmat{d.w_pool, Fi, Fi, Fi}, none, none, d.b_pool, nullptr,
                   saga_mat{b.z, V, Fi, b.ldz}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      op.msg = SAGA_MSG_COPY;
      op.reduce = SAGA_RED_MAX;
      in.src = saga_cmat{b.z, V, Fi, b.ldz};
      s = run_gather(p, op, in, saga_mat{b.z2, V, Fi, b.ldz2}, b.part, b.part_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      const char* w = static_cast<const char*>(d.w);
      g.mode = SAGA_GEMM_CONCAT;
      g.act = SAGA_ACT_NONE;
      s = run_gemm(g, x, saga_cmat{w, Fi, Fo, Fo}, saga_cmat{b.z2, V, Fi, b.ldz2},
                   saga_cmat{w + (size_t)Fi * Fo * es, Fi, Fo, Fo}, d.b, nullptr, out, b.gws, b.gws_bytes, st);
      if (s) return s;
      return stage_done(st, true);
    }
    case SAGA_LAYER_SAGE_LSTM: {
      // P = X W_ih + b_ih + b_hh; A = LSTM Gather; out = [X | A] W + b
      const int64_t H = d.hidden;
      g.mode = SAGA_GEMM_PLAIN;
      s = run_gemm(g, x, saga_cmat{d.w_ih, Fi, 4 * H, 4 * H}, none, none, d.b_ih, d.b_hh,
                   saga_mat{b.z, V, 4 * H, b.ldz}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      s = run_lstm(p, saga_cmat{b.z, V, 4 * H, b.ldz}, saga_cmat{d.w_hh, H, 4 * H, 4 * H},
                   saga_mat{b.z2, V, H, b.ldz2}, b.lstm_q, kLstmWs, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      const char* w = static_cast<const char*>(d.w);
      g.mode = SAGA_GEMM_CONCAT;
      s = run_gemm(g, x, saga_cmat{w, Fi, Fo, Fo}, saga_cmat{b.z2, V, H, b.ldz2},
                   saga_cmat{w + (size_t)Fi * Fo * 4, H, Fo, Fo}, d.b, nullptr, out, b.gws,
                   b.gws_bytes, st);
      if (s) return s;
      return stage_done(st, true);
    }
    case SAGA_LAYER_RGCN: {
      // T = pair rows x_u W_r; S = X W_self + b; out = act(S_v + sum_e norm_e T[pair_e])
      const saga_rel_plan& r = *d.rel;
      s = run_rel_transform(r, d.dtype, x, saga_cmat{d.w, r.num_rel * Fi, Fo, Fo},
                            saga_mat{b.z, r.max_pairs, Fo, b.ldz}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      g.mode = SAGA_GEMM_PLAIN;
      s = run_gemm(g, x, saga_cmat{d.w_self, Fi, Fo, Fo}, none, none, d.b, nullptr,
                   saga_mat{b.z2, V, Fo, b.ldz2}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      op.msg = SAGA_MSG_TYPED;
      op.reduce = SAGA_RED_SUM;
      op.act = d.act;
      in.src = saga_cmat{b.z, r.max_pairs, Fo, b.ldz};
      in.rel = &r;
      in.self = saga_cmat{b.z2, V, Fo, b.ldz2};
      s = run_gather(p, op, in, out, b.part, b.part_bytes, st);
      if (s) return s;
      return stage_done(st, true);
    }
    case SAGA_LAYER_GATED_GRU: {
      const int64_t F = Fi, Fe = d.edge_feat;
      g.mode = SAGA_GEMM_PLAIN;
      s = run_gemm(g, x, saga_cmat{d.w_e, F, F, F}, none, none, nullptr, nullptr,
                   saga_mat{b.z, V, F, b.ldz}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      s = run_gemm(g, x, saga_cmat{d.w_e + F * F, F, F, F}, none, none, nullptr, nullptr,
                   saga_mat{b.z2, V, F, b.ldz2}, b.gws, b.gws_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      op.msg = SAGA_MSG_GATED;
      op.reduce = SAGA_RED_SUM;
      in.src = x;
      in.gate_src = saga_cmat{b.z, V, F, b.ldz};
      in.gate_dst = saga_cmat{b.z2, V, F, b.ldz2};
      in.edge_feat = ef;
      if (ef.cols != Fe) return fail(SAGA_EINVAL, "edge_feat: %lld columns, desc says %d", (long long)ef.cols, d.edge_feat);
      in.w_edge = d.w_e + 2 * F * F;
      in.gate_bias = d.b_e;
      s = run_gather(p, op, in, saga_mat{b.z3, V, F, b.ldz3}, b.part, b.part_bytes, st);
      if (s) return s;
      if ((s = stage_done(st))) return s;
      g.mode = SAGA_GEMM_GRU;
      s = run_gemm(g, saga_cmat{b.z3, V, F, b.ldz3}, saga_cmat{d.w_ih, F, 3 * F, 3 * F}, x,
                   saga_cmat{d.w_hh, F, 3 * F, 3 * F}, d.b_ih, d.b_hh, out, b.gws, b.gws_bytes, st);
      if (s) return s;
      return stage_done(st, true);
    }
  }
  return fail(SAGA_EINVAL, "bad layer kind");
}

// ---------------------------------------------------------------------------
// Fixed device scratch of saga_scatter_apply_edge_gather_noalloc: the
// split-row partials live here instead of in a caller workspace.  Each GPU
// the library runs on holds its own copy until the process ends.  In host
// code the name `scratch` is a host-side stand-in, not a device address:
// kernels get the address noalloc_scratch() looked up for their device.
// ---------------------------------------------------------------------------
constexpr size_t kNoAllocScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices];

// Device address of `scratch` on device `dev`, looked up on first use with
// that device current and kept for the process.
hipError_t noalloc_scratch(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    hipError_t e = hipGetDevice(&cur);
    if (e != hipSuccess) return e;
    if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

const char* saga_status_str(saga_status s) {
  switch (s) {
    case SAGA_OK: return "ok";
    case SAGA_EINVAL: return "invalid argument";
    case SAGA_EGRAPH: return "invalid graph";
    case SAGA_EUNSUPPORTED: return "unsupported";
    case SAGA_EDEVICE: return "device error";
    case SAGA_EWORKSPACE: return "workspace too small";
    case SAGA_EINTERNAL: return "internal error";
  }
  return "unknown status";
}

const char* saga_last_error(void) { return g_err; }

const char* saga_version(void) { return "saga-mi355x 0.1 (gfx950)"; }

saga_status saga_sync_check(void* stream) {
  try {
    const hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return dev_fail(e, "stream");
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_plan_workspace_size(int32_t num_dst, int32_t num_src, int64_t num_edges,
                                     const saga_plan_opts* opts, size_t* bytes) {
  try {
    if (!bytes) return fail(SAGA_EINVAL, "bytes is null");
    int32_t T, B, c;
    saga_status s = resolve_opts(opts, num_dst, num_edges, &T, &B, &c);
    if (s) return s;
    saga::PlanLayout L;
    if (!saga::plan_layout(num_dst, num_src, num_edges, T, B, c, &L))
      return fail(SAGA_EINVAL, "graph sizes out of range (need 0 <= E < 2^31 and E + row_cost * segments < 2^31)");
    *bytes = L.total;
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status build_plan(int32_t num_dst, int32_t num_src, int64_t num_edges,
                       const int32_t* row_ptr, const int32_t* col_idx, const saga_plan_opts* opts,
                       void* workspace, size_t workspace_bytes, void* stream, void* order_stream,
                       void* fork_event, void* join_event, saga_plan* plan);

saga_status saga_plan_build(int32_t num_dst, int32_t num_src, int64_t num_edges,
                            const int32_t* row_ptr, const int32_t* col_idx,
                            const saga_plan_opts* opts, void* workspace, size_t workspace_bytes,
                            void* stream, saga_plan* plan) {
  return build_plan(num_dst, num_src, num_edges, row_ptr, col_idx, opts, workspace,
                    workspace_bytes, stream, nullptr, nullptr, nullptr, plan);
}

saga_status saga_plan_build_split(int32_t num_dst, int32_t num_src, int64_t num_edges,
                                  const int32_t* row_ptr, const int32_t* col_idx,
                                  const saga_plan_opts* opts, void* workspace,
                                  size_t workspace_bytes, void* stream, void* order_stream,
                                  void* fork_event, void* join_event, saga_plan* plan) {
  if (!order_stream || !fork_event || !join_event)
    return fail(SAGA_EINVAL, "plan split: order_stream, fork_event and join_event are required");
  if (order_stream == stream) return fail(SAGA_EINVAL, "plan split: order_stream is the stream");
  return build_plan(num_dst, num_src, num_edges, row_ptr, col_idx, opts, workspace,
                    workspace_bytes, stream, order_stream, fork_event, join_event, plan);
}

saga_status build_plan(int32_t num_dst, int32_t num_src, int64_t num_edges,
                       const int32_t* row_ptr, const int32_t* col_idx, const saga_plan_opts* opts,
                       void* workspace, size_t workspace_bytes, void* stream, void* order_stream,
                       void* fork_event, void* join_event, saga_plan* plan) {
  try {
    if (!plan) return fail(SAGA_EINVAL, "plan is null");
    int32_t T, B, c;
    saga_status s = resolve_opts(opts, num_dst, num_edges, &T, &B, &c);
    if (s) return s;
    saga::PlanLayout L;
    if (!saga::plan_layout(num_dst, num_src, num_edges, T, B, c, &L))
      return fail(SAGA_EINVAL, "graph sizes out of range");
    if (!row_ptr) return fail(SAGA_EINVAL, "row_ptr is null");
    if (num_edges > 0 && !col_idx) return fail(SAGA_EINVAL, "col_idx is null");
    if (!workspace || workspace_bytes < L.total)
      return fail(SAGA_EWORKSPACE, "plan workspace: need %zu bytes, got %zu", L.total, workspace_bytes);
    if ((uintptr_t)workspace % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
    char* w = static_cast<char*>(workspace);
    saga_plan p;
    memset(&p, 0, sizeof(p));
    p.num_dst = num_dst;
    p.num_src = num_src;
    p.num_edges = num_edges;
    p.row_ptr = row_ptr;
    p.col_idx = col_idx;
    p.seg_len = T;
    p.block_cost = B;
    p.row_cost = c;
    p.max_segments = L.max_segments;
    p.max_blocks = L.max_blocks;
    p.max_split = L.max_split;
    p.max_split_segments = L.max_split_segments;
    p.d_in = reinterpret_cast<int32_t*>(w + L.off_d_in);
    p.d_out = reinterpret_cast<int32_t*>(w + L.off_d_out);
    p.perm = reinterpret_cast<int32_t*>(w + L.off_perm);
    p.row_seg_first = reinterpret_cast<int32_t*>(w + L.off_first);
    p.seg_row = reinterpret_cast<int32_t*>(w + L.off_seg_row);
    p.seg_beg = reinterpret_cast<int32_t*>(w + L.off_seg_beg);
    p.seg_end = reinterpret_cast<int32_t*>(w + L.off_seg_end);
    p.block_ptr = reinterpret_cast<int32_t*>(w + L.off_block_ptr);
    p.counts = reinterpret_cast<int32_t*>(w + L.off_counts);
    p.scratch = w + L.off_scratch;
    p.scratch_bytes = L.scratch_bytes;
    hipError_t e = saga::launch_plan_build(p, L, static_cast<hipStream_t>(stream),
                                           static_cast<hipStream_t>(order_stream),
                                           static_cast<hipEvent_t>(fork_event),
                                           static_cast<hipEvent_t>(join_event));
    if (e != hipSuccess) return dev_fail(e, "plan launch");
    *plan = p;
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_plan_check(const saga_plan* plan, void* stream, saga_plan_counts* counts) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    hipStream_t st = static_cast<hipStream_t>(stream);
    int32_t h[saga::kCountSlots];
    hipError_t e = hipMemcpyAsync(h, plan->counts, sizeof(h), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return dev_fail(e, "plan check");
    if (counts) {
      counts->num_segments = h[saga::kNumSegments];
      counts->num_blocks = h[saga::kNumBlocks];
      counts->n_split = h[saga::kNSplit];
      counts->s_split = h[saga::kSSplit];
      counts->error_flags = h[saga::kErrFlags];
      counts->max_in_degree = h[saga::kMaxDegree];
    }
    const int f = h[saga::kErrFlags];
    if (f & saga::kErrInternal) return fail(SAGA_EINTERNAL, "plan builder invariant violated");
    if (f)
      return fail(SAGA_EGRAPH, "CSR invalid:%s%s%s%s", (f & 1) ? " row_ptr[0]!=0" : "",
                  (f & 2) ? " row_ptr decreasing" : "", (f & 4) ? " row_ptr[num_dst]!=num_edges" : "",
                  (f & 8) ? " col_idx out of range" : "");
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_gather_workspace_size(const saga_plan* plan, const saga_edge_op* op,
                                       int64_t feat, size_t* bytes) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !bytes) return fail(SAGA_EINVAL, "null argument");
    if (feat <= 0) return fail(SAGA_EINVAL, "feat must be > 0");
    return gather_ws_bytes(*plan, *op, feat, bytes) ? SAGA_EINTERNAL : ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_scatter_apply_edge_gather(const saga_plan* plan, const saga_edge_op* op,
                                           const saga_edge_inputs* in, saga_mat out,
                                           void* workspace, size_t workspace_bytes,
                                           void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !in) return fail(SAGA_EINVAL, "null argument");
    return run_gather(*plan, *op, *in, out, workspace, workspace_bytes,
                      static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_scatter_apply_edge_gather_noalloc(const saga_plan* plan, const saga_edge_op* op,
                                                   const saga_edge_inputs* in, saga_mat out,
                                                   void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !in) return fail(SAGA_EINVAL, "null argument");
    s = validate_edge_op(*plan, *op, *in, out);
    if (s) return s;
    size_t need = 0;
    gather_ws_bytes(*plan, *op, in->src.cols, &need);
    if (plan->max_split_segments > 0 && need > kNoAllocScratchBytes)
      return fail(SAGA_EUNSUPPORTED,
                  "noalloc gather: the split-row partials may need %zu bytes, the fixed scratch "
                  "holds %zu; use saga_scatter_apply_edge_gather with a workspace",
                  need, kNoAllocScratchBytes);
    hipStream_t st = static_cast<hipStream_t>(stream);
    int dev = -1;
    hipError_t e = st ? hipStreamGetDevice(st, &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return dev_fail(e, "noalloc gather: device of the stream");
    void* ws = nullptr;
    e = noalloc_scratch(dev, &ws);
    if (e != hipSuccess) return dev_fail(e, "noalloc gather: scratch address");
    return run_gather(*plan, *op, *in, out, ws, kNoAllocScratchBytes, st);
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_gather_transform_workspace_size(const saga_plan* plan, const saga_edge_op* op,
                                                 int64_t feat, size_t* bytes) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !bytes) return fail(SAGA_EINVAL, "null argument");
    if (feat <= 0) return fail(SAGA_EINVAL, "feat must be > 0");
    size_t part;
    gather_xf_ws_bytes(*plan, *op, feat, &part, bytes);
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_scatter_apply_edge_gather_transform(const saga_plan* plan, const saga_edge_op* op,
                                                     const saga_edge_inputs* in,
                                                     const saga_next_transform* next,
                                                     saga_mat out, void* workspace,
                                                     size_t workspace_bytes, void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !in || !next) return fail(SAGA_EINVAL, "null argument");
    return run_gather_transform(*plan, *op, *in, *next, out, workspace, workspace_bytes,
                                static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_unfused_workspace_size(const saga_plan* plan, const saga_edge_op* op,
                                        int64_t feat, size_t* bytes) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !bytes) return fail(SAGA_EINVAL, "null argument");
    if (feat <= 0) return fail(SAGA_EINVAL, "feat must be > 0");
    return unfused_ws_bytes(*plan, *op, feat, bytes) ? SAGA_EINTERNAL : ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_scatter_gather_unfused(const saga_plan* plan, const saga_edge_op* op,
                                        const saga_edge_inputs* in, saga_mat out,
                                        void* workspace, size_t workspace_bytes, void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!op || !in) return fail(SAGA_EINVAL, "null argument");
    return run_gather_unfused(*plan, *op, *in, out, workspace, workspace_bytes,
                              static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_lstm_gather_workspace_size(const saga_plan* plan, int64_t hidden,
                                            size_t* bytes) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!bytes) return fail(SAGA_EINVAL, "bytes is null");
    if (hidden != 32 && hidden != 64 && hidden != 128)
      return fail(SAGA_EUNSUPPORTED, "lstm gather: hidden size must be 32, 64 or 128");
    *bytes = kLstmWs;
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_lstm_gather(const saga_plan* plan, saga_cmat gates_x, saga_cmat w_hh,
                             saga_mat out, void* workspace, size_t workspace_bytes,
                             void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (plan->num_dst == 0) return ok();
    return run_lstm(*plan, gates_x, w_hh, out, workspace, workspace_bytes,
                    static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_rel_plan_workspace_size(const saga_plan* plan, int32_t num_rel, size_t* bytes) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!bytes) return fail(SAGA_EINVAL, "bytes is null");
    saga::RelLayout L;
    if (!saga::rel_layout(plan->num_src, plan->num_edges, num_rel, &L))
      return fail(SAGA_EINVAL, "num_rel must be in [1, %d] and pair rows below 2^31",
                  saga::kRelMaxRelations);
    *bytes = L.total;
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_rel_plan_build(const saga_plan* plan, const int32_t* etype, int32_t num_rel,
                                void* workspace, size_t workspace_bytes, void* stream,
                                saga_rel_plan* rel) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!rel) return fail(SAGA_EINVAL, "rel is null");
    if (plan->num_edges > 0 && !etype) return fail(SAGA_EINVAL, "etype is null");
    saga::RelLayout L;
    if (!saga::rel_layout(plan->num_src, plan->num_edges, num_rel, &L))
      return fail(SAGA_EINVAL, "num_rel must be in [1, %d] and pair rows below 2^31",
                  saga::kRelMaxRelations);
    if (!workspace || workspace_bytes < L.total)
      return fail(SAGA_EWORKSPACE, "rel plan workspace: need %zu bytes, got %zu", L.total,
                  workspace_bytes);
    if ((uintptr_t)workspace % 256 != 0) return fail(SAGA_EINVAL, "workspace must be 256-byte aligned");
    if (range_overlap(workspace, L.total, etype, (size_t)plan->num_edges * 4))
      return fail(SAGA_EINVAL, "workspace overlaps etype");
    char* w = static_cast<char*>(workspace);
    saga_rel_plan r;
    memset(&r, 0, sizeof(r));
    r.num_rel = num_rel;
    r.num_src = plan->num_src;
    r.num_edges = plan->num_edges;
    r.max_pairs = L.max_pairs;
    r.etype = etype;
    r.plan_counts = plan->counts;
    r.rel_ptr = reinterpret_cast<int32_t*>(w + L.off_rel_ptr);
    r.rel_count = reinterpret_cast<int32_t*>(w + L.off_rel_count);
    r.pair_src = reinterpret_cast<int32_t*>(w + L.off_pair_src);
    r.edge_pair = reinterpret_cast<int32_t*>(w + L.off_edge_pair);
    r.edge_norm = reinterpret_cast<float*>(w + L.off_edge_norm);
    r.counts = reinterpret_cast<int32_t*>(w + L.off_counts);
    r.scratch = w + L.off_scratch;
    r.scratch_bytes = L.scratch_bytes;
    hipError_t e = saga::launch_rel_build(*plan, r, L, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return dev_fail(e, "rel plan launch");
    *rel = r;
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_rel_plan_check(const saga_rel_plan* rel, void* stream, saga_rel_counts* counts) {
  try {
    if (!rel || !rel->counts || !rel->plan_counts) return fail(SAGA_EINVAL, "rel plan is not built");
    hipStream_t st = static_cast<hipStream_t>(stream);
    int32_t h[saga::kRelCountSlots], pc[saga::kCountSlots];
    hipError_t e = hipMemcpyAsync(h, rel->counts, sizeof(h), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipMemcpyAsync(pc, rel->plan_counts, sizeof(pc), hipMemcpyDeviceToHost, st);
    if (e == hipSuccess) e = hipStreamSynchronize(st);
    if (e != hipSuccess) return dev_fail(e, "rel plan check");
    if (counts) {
      counts->pair_rows = h[saga::kRelRows];
      counts->pairs = h[saga::kRelPairs];
      counts->error_flags = h[saga::kRelErr];
    }
    if (pc[saga::kErrFlags]) return fail(SAGA_EGRAPH, "the plan's CSR is invalid");
    if (h[saga::kRelErr]) return fail(SAGA_EGRAPH, "etype value outside [0, num_rel)");
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_rel_transform_workspace_size(const saga_rel_plan* rel, int32_t dtype,
                                              int64_t k, int64_t n, size_t* bytes) {
  try {
    if (!rel || !bytes) return fail(SAGA_EINVAL, "null argument");
    if (dtype != SAGA_F32 && dtype != SAGA_BF16) return fail(SAGA_EINVAL, "bad dtype");
    if (k <= 0 || n <= 0) return fail(SAGA_EINVAL, "k and n must be > 0");
    if (rel->num_rel < 1 || rel->num_rel > saga::kRelMaxRelations)
      return fail(SAGA_EINVAL, "rel plan is not built");
    *bytes = saga::gemm_grouped_workspace_bytes(dtype, rel->num_rel, n, k);
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_rel_transform(const saga_rel_plan* rel, int32_t dtype, saga_cmat x,
                               saga_cmat w, saga_mat out, void* workspace,
                               size_t workspace_bytes, void* stream) {
  try {
    if (!rel || !rel->counts || !rel->rel_ptr || !rel->pair_src || !rel->plan_counts)
      return fail(SAGA_EINVAL, "rel plan is not built");
    return run_rel_transform(*rel, dtype, x, w, out, workspace, workspace_bytes,
                             static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_lstm_gather_rows(const saga_plan* plan, int32_t perm_begin, int32_t perm_end,
                                  saga_cmat gates_x, saga_cmat w_hh, saga_mat out,
                                  void* workspace, size_t workspace_bytes, void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    return run_lstm(*plan, gates_x, w_hh, out, workspace, workspace_bytes,
                    static_cast<hipStream_t>(stream), perm_begin, perm_end);
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_apply_vertex_workspace_size(const saga_gemm_op* op, int64_t k, int64_t k2,
                                             int64_t n, size_t* bytes) {
  try {
    if (!op || !bytes) return fail(SAGA_EINVAL, "null argument");
    if (op->dtype != SAGA_F32 && op->dtype != SAGA_BF16) return fail(SAGA_EINVAL, "bad dtype");
    if (op->mode < SAGA_GEMM_PLAIN || op->mode > SAGA_GEMM_GRU) return fail(SAGA_EINVAL, "bad mode");
    if (k <= 0 || n <= 0 || (op->mode != SAGA_GEMM_PLAIN && k2 <= 0))
      return fail(SAGA_EINVAL, "k, n (and k2 for concat/GRU) must be > 0");
    *bytes = gemm_ws_bytes(*op, k, k2, n);
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_apply_vertex(const saga_gemm_op* op, saga_cmat a, saga_cmat w, saga_cmat a2,
                              saga_cmat w2, const float* bias, const float* bias2, saga_mat out,
                              void* workspace, size_t workspace_bytes, void* stream) {
  try {
    if (!op) return fail(SAGA_EINVAL, "op is null");
    return run_gemm(*op, a, w, a2, w2, bias, bias2, out, workspace, workspace_bytes,
                    static_cast<hipStream_t>(stream));
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_layer_workspace_size(const saga_plan* plan, const saga_layer_desc* desc,
                                      size_t* bytes) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!desc || !bytes) return fail(SAGA_EINVAL, "null argument");
    s = layer_check_desc(*plan, *desc);
    if (s) return s;
    LayerBufs b;
    *bytes = layer_carve(*plan, *desc, nullptr, &b);
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_trace_stages(void* const* events, int32_t n_events, int32_t markers) {
  try {
    if (n_events < 0 || (n_events > 0 && !events))
      return fail(SAGA_EINVAL, "trace: %d events at %p", n_events, (const void*)events);
    for (int32_t i = 0; i < n_events; ++i)
      if (!events[i]) return fail(SAGA_EINVAL, "trace: event %d is null", i);
    g_stage_events.assign(reinterpret_cast<const hipEvent_t*>(events),
                          reinterpret_cast<const hipEvent_t*>(events) + n_events);
    g_stage_markers = markers ? 1 : 0;
    g_stage_next = 0;
    return ok();
  } catch (...) {
    return fail(SAGA_EINTERNAL, "exception");
  }
}

saga_status saga_layer(const saga_plan* plan, const saga_layer_desc* desc, saga_cmat x,
                       saga_cmat edge_feat, saga_mat out, void* workspace, size_t workspace_bytes,
                       void* stream) {
  try {
    saga_status s = check_plan(plan);
    if (s) return s;
    if (!desc) return fail(SAGA_EINVAL, "desc is null");
    s = run_layer(*plan, *desc, x, edge_feat, out, workspace, workspace_bytes,
                  static_cast<hipStream_t>(stream));
    stage_ranges_close();
    return s;
  } catch (...) {
    stage_ranges_close();
    return fail(SAGA_EINTERNAL, "exception");
  }
}

}  // extern "C"
