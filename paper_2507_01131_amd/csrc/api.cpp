// C ABI of the CP tensor-product layer: argument validation, workspace
// layout, launch sequence and status reporting.  No allocation happens here:
// every scratch buffer is carved from the caller's workspace.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "api_internal.h"
#include "kernels.h"
#include "tdn.h"


namespace {

thread_local int32_t g_last_hip = 0;
// set while a call must not create timing events (tdn_cp_tp_forward_noalloc)
thread_local bool g_untimed = false;

size_t al(size_t b) { return (b + 255) & ~size_t(255); }

tdn_status hip_fail(hipError_t e) {
  g_last_hip = int32_t(e);
  return TDN_ERR_HIP;
}

#define TDN_HIP(expr)                           \
  do {                                          \
    hipError_t e_ = (expr);                     \
    if (e_ != hipSuccess) return hip_fail(e_);  \
  } while (0)

int dim_of(int L) { return (L + 1) * (L + 1); }

// Ranks: the edge kernels take at most kChunkR; larger ranks (up to
// kMaxRank, e.g. the exact rank d^2 construction of Thm. 2) run as chunks of
// consecutive 32-rank tiles, balanced, whose per-node results are summed in
// chunk order (the layer is linear in each rank component).
constexpr int kChunkR = 256;
constexpr int kMaxRank = 4096;
int rank_chunks(int R) { return (R + kChunkR - 1) / kChunkR; }
void chunk_range(int R, int c, int nch, int* r0, int* n) {
  const int tiles = (R + 31) / 32, per = (tiles + nch - 1) / nch;
  *r0 = std::min(R, c * per * 32);
  *n = std::min(per * 32, R - *r0);
}
tdn_problem chunk_problem(const tdn_problem& p, int c) {
  tdn_problem q = p;
  int r0 = 0, n = p.R;
  chunk_range(p.R, c, rank_chunks(p.R), &r0, &n);
  q.R = n;
  return q;
}

tdn_status check_problem(const tdn_problem* p) {
  if (!p) return TDN_ERR_NULL_POINTER;
  if (p->feat_dtype != TDN_F32 && p->feat_dtype != TDN_BF16) return TDN_ERR_BAD_DTYPE;
  if (p->L < 0 || p->L > 6) return TDN_ERR_BAD_SHAPE;
  if (p->C < 16 || p->C > 256 || p->C % 16 != 0) return TDN_ERR_BAD_SHAPE;
  if (p->R < 1 || p->R > kMaxRank) return TDN_ERR_BAD_SHAPE;
  if (p->n_nodes < 0 || p->n_edges < 0) return TDN_ERR_BAD_SHAPE;
  if (p->n_edges > 0 && p->n_nodes == 0) return TDN_ERR_BAD_SHAPE;
  if (p->n_radial < 2 || p->n_radial > 16) return TDN_ERR_BAD_SHAPE;
  if (!(p->r_cut > 0.f) || !std::isfinite(p->r_cut)) return TDN_ERR_BAD_SHAPE;
  if (int64_t(p->n_nodes) * dim_of(p->L) * p->C >= (int64_t(1) << 40)) return TDN_ERR_BAD_SHAPE;
  if (int64_t(p->n_nodes) * dim_of(p->L) >= (int64_t(1) << 31) - 1) return TDN_ERR_BAD_SHAPE;
  if (p->edges_sorted != 0 && p->edges_sorted != 1) return TDN_ERR_BAD_SHAPE;
  return TDN_OK;
}

// 16-bit parts per feature of the edge pass: the fp16 two-part split of
// fp32 features, or the bf16 features themselves
int feature_parts(const tdn_problem& p) { return p.feat_dtype == TDN_BF16 ? 1 : 2; }

// features of the edge pass in MFMA operand blocks, then their row scales
size_t xs_bytes(const tdn_problem& p) {
  return size_t(p.n_nodes) * ((p.C + 31) / 32 * 32) * feature_parts(p) * tdn::edge_kpad(dim_of(p.L)) * 2;
}
size_t xt_bytes(const tdn_problem& p) { return al(xs_bytes(p)) + size_t(p.n_nodes) * 4; }
float* row_scales(const tdn_problem& p, void* xt) {
  return reinterpret_cast<float*>(static_cast<char*>(xt) + al(xs_bytes(p)));
}
// the same region holds, in the backward, x blocked over channels for
// the destination-side kernel
// x in the direct destination kernel's operand blocks (d > 32), then its row
// scales
size_t xd_bytes(const tdn_problem& p) {
  return size_t(p.n_nodes) * dim_of(p.L) * feature_parts(p) * tdn::bwd_direct_cpad(p.C) * 2;
}
size_t xc_bytes(const tdn_problem& p) {
  return size_t(p.n_nodes) * dim_of(p.L) * feature_parts(p) * tdn::bwd_dst_cpad(p.C, p.feat_dtype == TDN_BF16) * 2;
}
size_t xt_xc_bytes(const tdn_problem& p) {
  const size_t xc = al(xc_bytes(p)) + size_t(p.n_nodes) * 4;
  const size_t xd = al(xd_bytes(p)) + size_t(p.n_nodes) * 4;
  return std::max(xt_bytes(p), std::max(xc, xd));
}

// the output factor's epilogue operand blocks and scale, then the partial
// slots of the edge pass (two [d, C] rows per edge range)
size_t ef_pad_bytes(const tdn_problem& p) { return al(tdn::edge_ef_bytes(dim_of(p.L), p.R)); }
size_t partial_bytes_one(const tdn_problem& p) {
  const bool bf16 = p.feat_dtype == TDN_BF16;
  int n_range = tdn::edge_plan(p.L, p.R, p.C, p.n_radial, bf16, p.n_edges).n_range;
  if (!bf16 && p.L >= 2 && p.L <= 4)  // the three-input product's plan may use more ranges
    n_range = std::max(n_range, tdn::edge_plan(p.L, p.R, p.C, p.n_radial, false, p.n_edges, true).n_range);
  return ef_pad_bytes(p) + size_t(n_range) * 2 * dim_of(p.L) * p.C * 4;
}
// the largest over the problem's rank chunks
size_t partial_bytes(const tdn_problem& p) {
  size_t m = 0;
  for (int c = 0; c < rank_chunks(p.R); ++c) m = std::max(m, partial_bytes_one(chunk_problem(p, c)));
  return m;
}
// rank chunks: the chunk's factor and radial-weight columns
size_t slice_bytes(const tdn_problem& p) {
  return rank_chunks(p.R) > 1 ? size_t(3 * dim_of(p.L) + p.n_radial) * kChunkR * 4 : 0;
}

struct FwdLayout {
  size_t z, xt, part, sort, wp, fsl, ztmp, flags, total;
};
FwdLayout fwd_layout(const tdn_problem& p) {
  FwdLayout f{};
  const size_t ndc = size_t(p.n_nodes) * dim_of(p.L) * p.C * 4;
  size_t o = 0;
  f.z = o;
  o += al(ndc);
  f.xt = o;
  o += al(xt_bytes(p));
  f.part = o;
  o += al(partial_bytes(p));
  f.sort = o;
  o += al(p.edges_sorted ? 0 : tdn::sort_plan(p.n_nodes, p.n_edges).bytes);
  f.wp = o;
  o += al(tdn::node_gemm_ws_bytes(p.C));
  f.fsl = o;  // rank chunks: factor columns and a second Z for the chunks after the first
  o += al(slice_bytes(p));
  f.ztmp = o;
  o += rank_chunks(p.R) > 1 ? al(ndc) : 0;
  f.flags = o;
  o += 256;
  f.total = o;
  return f;
}

struct BwdLayout {
  size_t gz, z, xt, part, parts, perm_src, off_src, sort, wp, drho, wrad_part, gv, fsl, gtmp, grtmp, bt, gzc, flags,
      total;
};
BwdLayout bwd_layout(const tdn_problem& p) {
  BwdLayout b{};
  const size_t ndc = size_t(p.n_nodes) * dim_of(p.L) * p.C * 4;
  size_t o = 0;
  b.gz = o;
  o += al(ndc);
  b.z = o;
  o += al(ndc);
  b.xt = o;
  o += al(xt_xc_bytes(p));
  b.part = o;
  o += al(partial_bytes(p));
  b.parts = o;
  o += al(size_t(tdn::gram_parts(p.n_nodes * dim_of(p.L), p.C)) * p.C * p.C * 4);
  b.perm_src = o;
  o += al(size_t(p.n_edges) * 4);
  b.off_src = o;
  o += al(size_t(p.n_nodes + 1) * 4);
  b.sort = o;
  o += al(tdn::sort_plan(p.n_nodes, p.n_edges).bytes);
  b.wp = o;
  o += al(tdn::node_gemm_ws_bytes(p.C));
  const int rc = chunk_problem(p, 0).R;  // the largest rank chunk (p.R when not chunked)
  b.drho = o;  // radial-weight gradient: dL/drho per edge, block partials, and a
  o += al(size_t(p.n_edges) * rc * 4);  // grad_edge_vec stand-in when only grad_radial_w is asked for
  b.wrad_part = o;  // partials of the radial_grad kernel or of the range kernel's workgroups
  o += al(size_t(std::max(tdn::radial_grad_blocks(p.n_edges), 2 * tdn::device_cus())) * p.n_radial * rc * 4);
  b.gv = o;
  o += al(size_t(p.n_edges) * 12);
  const bool chunked = rank_chunks(p.R) > 1;
  b.fsl = o;  // rank chunks: factor columns, a chunk's grad_x or grad_edge_vec, a chunk's radial gradient
  o += al(slice_bytes(p));
  b.gtmp = o;
  o += chunked ? al(std::max(ndc, size_t(p.n_edges) * 12)) : 0;
  b.grtmp = o;
  o += chunked ? al(size_t(p.n_radial) * rc * 4) : 0;
  b.bt = o;  // direct destination kernel (d > 32): B^T and Wrad^T of a rank chunk
  o += dim_of(p.L) > 32 ? al(size_t(dim_of(p.L) + p.n_radial) * rc * 4) : 0;
  b.gzc = o;  // split form of the destination kernel: Gz in the layout of xc, then its row scales
  o += tdn::bwd_dst_split(p.L, p.C, p.feat_dtype == TDN_BF16) ? al(xc_bytes(p)) + al(size_t(p.n_nodes) * 4) : 0;
  b.flags = o;
  o += 256;
  b.total = o;
  return b;
}

tdn_status check_device() {
  // an error left pending by earlier, unrelated HIP work must not be
  // reported as this call's launch failure
  (void)hipGetLastError();
  int dev = 0;
  TDN_HIP(hipGetDevice(&dev));
  static std::mutex mu;
  static std::map<int, bool> known;
  std::lock_guard<std::mutex> lk(mu);
  auto it = known.find(dev);
  if (it == known.end()) {
    hipDeviceProp_t prop;
    TDN_HIP(hipGetDeviceProperties(&prop, dev));
    it = known.emplace(dev, std::strncmp(prop.gcnArchName, "gfx950", 6) == 0).first;
  }
  return it->second ? TDN_OK : TDN_ERR_UNSUPPORTED_DEVICE;
}

// --------------------------------------------------------------- timing
struct Timer {
  bool on = false;
  std::mutex mu;
  std::map<std::string, std::vector<std::pair<hipEvent_t, hipEvent_t>>> pending;
  std::map<std::string, std::pair<double, int>> done;
};
Timer& timer() {
  static Timer t;
  return t;
}

class Timed {
 public:
  Timed(const char* name, hipStream_t s) : name_(name), s_(s) {
    if (g_untimed) return;
    Timer& t = timer();
    std::lock_guard<std::mutex> lk(t.mu);
    if (!t.on) return;
    if (hipEventCreate(&a_) != hipSuccess || hipEventCreate(&b_) != hipSuccess) return;
    hipEventRecord(a_, s_);
  }
  ~Timed() {
    if (!a_ || !b_) return;
    hipEventRecord(b_, s_);
    Timer& t = timer();
    std::lock_guard<std::mutex> lk(t.mu);
    t.pending[name_].emplace_back(a_, b_);
  }

 private:
  const char* name_;
  hipStream_t s_;
  hipEvent_t a_ = nullptr, b_ = nullptr;
};

tdn_status run_validation(const tdn_problem& p, const int32_t* edge_index, const float* edge_vec, char* ws,
                          size_t flags_off, int check_sorted, hipStream_t s) {
  int32_t* flags = reinterpret_cast<int32_t*>(ws + flags_off);
  TDN_HIP(tdn::launch_validate(p.n_nodes, p.n_edges, edge_index, edge_vec, check_sorted, flags, s));
  int32_t host[4] = {0, 0, 0, 0};
  TDN_HIP(hipMemcpyAsync(host, flags, sizeof(host), hipMemcpyDeviceToHost, s));
  TDN_HIP(hipStreamSynchronize(s));
  if (host[0]) return TDN_ERR_INDEX_OUT_OF_RANGE;
  if (host[1]) return TDN_ERR_NOT_SORTED;
  if (host[2]) return TDN_ERR_DEGENERATE_EDGE;
  return TDN_OK;
}

tdn::EdgeArgs edge_args(const tdn_problem& p, const int32_t* offsets, const int32_t* perm, const int32_t* gather,
                        const int32_t* key, const float* edge_vec, const float* KF, const float* EF, const float* B,
                        const float* radial_w, const void* feat, float* out, float* partial, bool t3 = false) {
  tdn::EdgeArgs a{};
  a.n_seg = p.n_nodes;
  a.E = p.n_edges;
  a.L = p.L;
  a.d = dim_of(p.L);
  a.C = p.C;
  a.R = p.R;
  a.n_radial = p.n_radial;
  a.sigma = p.r_cut / float(p.n_radial - 1);
  a.offsets = offsets;
  a.perm = perm;
  a.gather = gather;
  a.key = key;
  a.edge_vec = edge_vec;
  a.KF = KF;
  a.EF = EF;
  a.Bf = B;
  a.radial_w = radial_w;
  a.feat = feat;
  a.out = out;
  const tdn::EdgePlan pl = tdn::edge_plan(p.L, p.R, p.C, p.n_radial, p.feat_dtype == TDN_BF16, p.n_edges, t3);
  a.n_range = pl.n_range;
  a.pieces_per_block = pl.per_block;
  a.ef_ops = partial;
  a.ef_scale = partial ? reinterpret_cast<float*>(reinterpret_cast<char*>(partial) +
                                                 tdn::edge_ef_bytes(dim_of(p.L), p.R) - 256)
                       : nullptr;
  a.parts = feature_parts(p);
  a.row_scale = a.parts == 2 ? row_scales(p, const_cast<void*>(feat)) : nullptr;
  a.partial = partial ? reinterpret_cast<float*>(reinterpret_cast<char*>(partial) + ef_pad_bytes(p)) : nullptr;
  return a;
}

// Features of the CP edge pass: the packed fp16 split of fp32 features, or
// the bf16 operand blocks (bf16 problems; an fp32 input is rounded).
hipError_t edge_features(const tdn_problem& p, const void* x, bool x_is_f32, void* xt, hipStream_t s) {
  if (feature_parts(p) == 2)
    return tdn::launch_feature_layout_packed(p.n_nodes, dim_of(p.L), p.C, static_cast<const float*>(x), xt,
                                             row_scales(p, xt), s);
  return tdn::launch_feature_layout(p.n_nodes, dim_of(p.L), p.C, x, x_is_f32, 1, xt, nullptr, s);
}

// The edge pass out[seg] = per-segment EF diag(g) KF^T feat sums over all R
// ranks: one launch when R <= kChunkR, otherwise one per rank chunk (the
// chunk's columns of KF, EF, B and radial_w cut into fsl), the chunks after
// the first written to otmp and added into out in chunk order.  feat must
// already be laid out (edge_features).
hipError_t edge_pass_ranks(const tdn_problem& p, const int32_t* offsets, const int32_t* perm, const int32_t* gather,
                           const int32_t* key, const float* edge_vec, const float* KF, const float* EF,
                           const float* B, const float* radial_w, const void* feat, float* out, float* partial,
                           float* fsl, float* otmp, hipStream_t s, bool atomic = false) {
  const int nch = rank_chunks(p.R);
  if (nch == 1) {
    const tdn::EdgeArgs a = edge_args(p, offsets, perm, gather, key, edge_vec, KF, EF, B, radial_w, feat, out, partial);
    return atomic ? tdn::launch_cp_edge_atomic(a, s) : tdn::launch_cp_edge(a, s);
  }
  if (atomic) return hipErrorInvalidValue;
  const int d = dim_of(p.L);
  float *sK = fsl, *sE = fsl + size_t(d) * kChunkR, *sB = fsl + size_t(2 * d) * kChunkR;
  float* sW = fsl + size_t(3 * d) * kChunkR;
  for (int c = 0; c < nch; ++c) {
    int r0 = 0, n = 0;
    chunk_range(p.R, c, nch, &r0, &n);
    tdn_problem pc = p;
    pc.R = n;
    hipError_t e = tdn::launch_slice_cols(d, p.R, r0, n, KF, sK, s);
    if (e == hipSuccess) e = tdn::launch_slice_cols(d, p.R, r0, n, EF, sE, s);
    if (e == hipSuccess) e = tdn::launch_slice_cols(d, p.R, r0, n, B, sB, s);
    if (e == hipSuccess) e = tdn::launch_slice_cols(p.n_radial, p.R, r0, n, radial_w, sW, s);
    if (e != hipSuccess) return e;
    float* dst = c == 0 ? out : otmp;
    const tdn::EdgeArgs a = edge_args(pc, offsets, perm, gather, key, edge_vec, sK, sE, sB, sW, feat, dst, partial);
    e = tdn::launch_cp_edge(a, s);
    if (e == hipSuccess && c > 0) e = tdn::launch_accumulate(size_t(p.n_nodes) * d * p.C, otmp, out, s);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

// The forward edge pass Z = per-node D diag(g) A^T x sums, for either
// feature dtype (features laid out into xt first).
hipError_t forward_edge_pass(const tdn_problem& p, const int32_t* offsets, const int32_t* perm, const int32_t* src,
                             const int32_t* dst, const float* edge_vec, const float* A, const float* B, const float* D,
                             const float* radial_w, const void* x, void* xt, float* partial, float* Z, float* fsl,
                             float* ztmp, hipStream_t s, bool atomic = false) {
  {
    Timed t("feature_layout", s);
    hipError_t e = edge_features(p, x, p.feat_dtype == TDN_F32, xt, s);
    if (e != hipSuccess) return e;
  }
  Timed t(atomic ? "cp_edge_fwd_atomic" : "cp_edge_fwd", s);
  return edge_pass_ranks(p, offsets, perm, src, dst, edge_vec, A, D, B, radial_w, xt, Z, partial, fsl, ztmp, s,
                         atomic);
}

}  // namespace

extern "C" {

const char* tdn_status_string(tdn_status s) {
  switch (s) {
    case TDN_OK: return "ok";
    case TDN_ERR_NULL_POINTER: return "null pointer";
    case TDN_ERR_BAD_SHAPE: return "bad shape";
    case TDN_ERR_BAD_DTYPE: return "bad dtype";
    case TDN_ERR_WORKSPACE_TOO_SMALL: return "workspace too small";
    case TDN_ERR_INDEX_OUT_OF_RANGE: return "edge index out of range";
    case TDN_ERR_NOT_SORTED: return "edges not sorted by destination";
    case TDN_ERR_DEGENERATE_EDGE: return "zero-length or non-finite edge vector";
    case TDN_ERR_UNSUPPORTED_DEVICE: return "unsupported device (needs gfx950)";
    case TDN_ERR_HIP: return "HIP error";
    case TDN_ERR_BAD_GEOMETRY: return "invalid graph_ptr, position or periodic box";
    case TDN_ERR_EDGE_CAPACITY: return "edge buffers smaller than the edge count";
    case TDN_ERR_NEIGHBOUR_LIMIT: return "more than 2048 neighbours of one atom within the cutoff";
    case TDN_ERR_SCRATCH_LIMIT:
      return "the problem needs more workspace than the no-allocation entry point's fixed scratch area holds";
  }
  return "unknown status";
}

int32_t tdn_last_hip_error(void) { return g_last_hip; }

tdn_status tdn_workspace_size(const tdn_problem* p, size_t* fwd_bytes, size_t* bwd_bytes) {
  const tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (fwd_bytes) *fwd_bytes = fwd_layout(*p).total;
  if (bwd_bytes) *bwd_bytes = bwd_layout(*p).total;
  return TDN_OK;
}

namespace {
tdn_status forward_impl(const tdn_problem* p, const void* x, const float* edge_vec, const int32_t* edge_index,
                        const float* A, const float* B, const float* D, const void* W, const float* radial_w,
                        float* out, float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                        size_t workspace_bytes, hipStream_t stream, bool atomic) {
  tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (atomic && p->feat_dtype != TDN_F32) return TDN_ERR_BAD_DTYPE;
  if (atomic && (p->L < 2 || p->L > 4 || p->R > kChunkR)) return TDN_ERR_BAD_SHAPE;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C;
  if (!A || !B || !D || !W || !radial_w || !offsets || !workspace) return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const FwdLayout lay = fwd_layout(*p);
  if (workspace_bytes < lay.total) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, p->edges_sorted, stream);
    if (st != TDN_OK) return st;
  }
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  {
    Timed t("sort", stream);
    if (p->edges_sorted || E == 0)
      TDN_HIP(tdn::launch_offsets_presorted(N, E, dst, perm, offsets, stream));
    else
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), dst, 1, perm, offsets, ws + lay.sort, stream));
  }
  if (N == 0) return TDN_OK;
  float* Z = z_save ? z_save : reinterpret_cast<float*>(ws + lay.z);
  const bool bf16 = p->feat_dtype == TDN_BF16;
  TDN_HIP(forward_edge_pass(*p, offsets, perm, src, dst, edge_vec, A, B, D, radial_w, x, ws + lay.xt,
                            reinterpret_cast<float*>(ws + lay.part), Z, reinterpret_cast<float*>(ws + lay.fsl),
                            reinterpret_cast<float*>(ws + lay.ztmp), stream, atomic));
  {
    Timed t("node_gemm", stream);
    TDN_HIP(tdn::launch_node_gemm(N * d, C, Z, W, bf16, 0, out, ws + lay.wp, stream));
  }
  return TDN_OK;
}
}  // namespace

tdn_status tdn_cp_tp_forward(const tdn_problem* p, const void* x, const float* edge_vec, const int32_t* edge_index,
                             const float* A, const float* B, const float* D, const void* W, const float* radial_w,
                             float* out, float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                             size_t workspace_bytes, hipStream_t stream) {
  return forward_impl(p, x, edge_vec, edge_index, A, B, D, W, radial_w, out, z_save, perm, offsets, workspace,
                      workspace_bytes, stream, false);
}

tdn_status tdn_ablation_forward_atomics(const tdn_problem* p, const void* x, const float* edge_vec,
                                        const int32_t* edge_index, const float* A, const float* B, const float* D,
                                        const void* W, const float* radial_w, float* out, float* z_save,
                                        int32_t* perm, int32_t* offsets, void* workspace, size_t workspace_bytes,
                                        hipStream_t stream) {
  return forward_impl(p, x, edge_vec, edge_index, A, B, D, W, radial_w, out, z_save, perm, offsets, workspace,
                      workspace_bytes, stream, true);
}

namespace {
// The measurement ablations' extra workspace after the forward's: the
// per-workgroup factor copies, or the harmonics table.
size_t abl_extra_bytes(const tdn_problem& p, int variant) {
  if (variant == tdn::kAblFactorsGlobal) {
    const tdn::EdgePlan pl = tdn::edge_plan(p.L, p.R, p.C, p.n_radial, false, p.n_edges);
    return al(tdn::edge_abl_fa_bytes(p.L, p.R, p.C, pl.n_range, pl.per_block));
  }
  if (variant == tdn::kAblYTable) return al(size_t(p.n_edges) * dim_of(p.L) * 4);
  return 0;
}
tdn_status check_ablation(const tdn_problem* p, int32_t variant) {
  const tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (variant != tdn::kAblFactorsGlobal && variant != tdn::kAblYTable && variant != tdn::kAblValu)
    return TDN_ERR_BAD_SHAPE;
  if (p->feat_dtype != TDN_F32) return TDN_ERR_BAD_DTYPE;
  if (p->L < 2 || p->L > 4 || p->R > kChunkR) return TDN_ERR_BAD_SHAPE;
  if (variant == tdn::kAblValu && (p->R > 128 || p->C > 128)) return TDN_ERR_BAD_SHAPE;
  return TDN_OK;
}
}  // namespace

tdn_status tdn_ablation_workspace_size(const tdn_problem* p, int32_t variant, size_t* bytes) {
  const tdn_status st = check_ablation(p, variant);
  if (st != TDN_OK) return st;
  if (!bytes) return TDN_ERR_NULL_POINTER;
  *bytes = fwd_layout(*p).total + abl_extra_bytes(*p, variant);
  return TDN_OK;
}

tdn_status tdn_ablation_forward(const tdn_problem* p, int32_t variant, const void* x, const float* edge_vec,
                                const int32_t* edge_index, const float* A, const float* B, const float* D,
                                const void* W, const float* radial_w, float* out, float* z_save, int32_t* perm,
                                int32_t* offsets, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tdn_status st = check_ablation(p, variant);
  if (st != TDN_OK) return st;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C;
  if (!A || !B || !D || !W || !radial_w || !offsets || !workspace) return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const FwdLayout lay = fwd_layout(*p);
  if (workspace_bytes < lay.total + abl_extra_bytes(*p, variant)) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, p->edges_sorted, stream);
    if (st != TDN_OK) return st;
  }
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  {
    Timed t("sort", stream);
    if (p->edges_sorted || E == 0)
      TDN_HIP(tdn::launch_offsets_presorted(N, E, dst, perm, offsets, stream));
    else
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), dst, 1, perm, offsets, ws + lay.sort, stream));
  }
  if (N == 0) return TDN_OK;
  float* Z = z_save ? z_save : reinterpret_cast<float*>(ws + lay.z);
  float* partial = reinterpret_cast<float*>(ws + lay.part);
  tdn::EdgeArgs a = edge_args(*p, offsets, perm, src, dst, edge_vec, A, D, B, radial_w, ws + lay.xt, Z, partial);
  if (variant != tdn::kAblValu) {
    Timed t("feature_layout", stream);
    TDN_HIP(edge_features(*p, x, true, ws + lay.xt, stream));
  }
  if (variant == tdn::kAblFactorsGlobal) a.fa_global = ws + lay.total;
  if (variant == tdn::kAblYTable && E > 0) {
    float* yt = reinterpret_cast<float*>(ws + lay.total);
    Timed t("sh_table", stream);
    TDN_HIP(tdn::launch_sh(p->L, E, edge_vec, yt, nullptr, stream));
    a.y_table = yt;
  }
  {
    Timed t("cp_edge_fwd_ablation", stream);
    TDN_HIP(tdn::launch_cp_edge_ablation(a, variant, static_cast<const float*>(x), stream));
  }
  {
    Timed t("node_gemm", stream);
    TDN_HIP(tdn::launch_node_gemm(N * d, C, Z, W, false, 0, out, ws + lay.wp, stream));
  }
  return TDN_OK;
}

namespace {
// The attention block's workspace after the forward's: Pt and Ps [N, F], the
// weights by sorted position [E, H].
size_t att_extra_bytes(const tdn_problem& p, int H, int F) {
  return al(size_t(p.n_nodes) * F * 4) * 2 + al(size_t(p.n_edges) * H * 4);
}
tdn_status check_attention(const tdn_problem* p, int32_t n_heads, int32_t n_hidden) {
  const tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (p->feat_dtype != TDN_F32) return TDN_ERR_BAD_DTYPE;
  if (p->L < 1 || p->L > 4 || p->R > kChunkR || n_heads < 1 || n_heads > 8 || p->C % (32 * n_heads) != 0 ||
      n_hidden < 1 || n_hidden > 64)
    return TDN_ERR_BAD_SHAPE;
  return TDN_OK;
}
}  // namespace

tdn_status tdn_attention_workspace_size(const tdn_problem* p, int32_t n_heads, int32_t n_hidden, size_t* bytes) {
  const tdn_status st = check_attention(p, n_heads, n_hidden);
  if (st != TDN_OK) return st;
  if (!bytes) return TDN_ERR_NULL_POINTER;
  *bytes = fwd_layout(*p).total + att_extra_bytes(*p, n_heads, n_hidden);
  return TDN_OK;
}

tdn_status tdn_attention_forward(const tdn_problem* p, int32_t n_heads, int32_t n_hidden, const float* x,
                                 const float* edge_vec, const int32_t* edge_index, const float* A, const float* B,
                                 const float* D, const float* W, const float* radial_w, const float* att_w1,
                                 const float* att_w2, float* out, float* alpha, float* z_save, int32_t* perm,
                                 int32_t* offsets, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tdn_status st = check_attention(p, n_heads, n_hidden);
  if (st != TDN_OK) return st;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C, F = n_hidden, H = n_heads;
  if (!A || !B || !D || !W || !radial_w || !att_w1 || !att_w2 || !offsets || !workspace) return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const FwdLayout lay = fwd_layout(*p);
  if (workspace_bytes < lay.total + att_extra_bytes(*p, H, F)) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, p->edges_sorted, stream);
    if (st != TDN_OK) return st;
  }
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  {
    Timed t("sort", stream);
    if (p->edges_sorted || E == 0)
      TDN_HIP(tdn::launch_offsets_presorted(N, E, dst, perm, offsets, stream));
    else
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), dst, 1, perm, offsets, ws + lay.sort, stream));
  }
  if (N == 0) return TDN_OK;
  float* Pt = reinterpret_cast<float*>(ws + lay.total);
  float* Ps = reinterpret_cast<float*>(ws + lay.total + al(size_t(N) * F * 4));
  float* al_sorted = reinterpret_cast<float*>(ws + lay.total + 2 * al(size_t(N) * F * 4));
  {
    Timed t("attention_weights", stream);
    TDN_HIP(tdn::launch_att_node(N, d, C, F, x, att_w1, Pt, Ps, stream));
    TDN_HIP(tdn::launch_att_alpha(N, C, F, H, p->n_radial, p->r_cut / float(p->n_radial - 1), offsets, perm, src,
                                  edge_vec, Pt, Ps, att_w1, att_w2, al_sorted, alpha, stream));
  }
  float* Z = z_save ? z_save : reinterpret_cast<float*>(ws + lay.z);
  {
    Timed t("feature_layout", stream);
    TDN_HIP(edge_features(*p, x, true, ws + lay.xt, stream));
  }
  {
    Timed t("cp_edge_fwd_att", stream);
    tdn::EdgeArgs a = edge_args(*p, offsets, perm, src, dst, edge_vec, A, D, B, radial_w, ws + lay.xt, Z,
                                reinterpret_cast<float*>(ws + lay.part));
    a.alpha = al_sorted;
    a.n_heads = H;
    TDN_HIP(tdn::launch_cp_edge_att(a, stream));
  }
  {
    Timed t("node_gemm", stream);
    TDN_HIP(tdn::launch_node_gemm(N * d, C, Z, W, false, 0, out, ws + lay.wp, stream));
  }
  return TDN_OK;
}

tdn_status tdn_cp_tp3_forward(const tdn_problem* p, const void* x, const float* edge_vec, const int32_t* edge_index,
                              const float* A, const float* A2, const float* B, const float* D, const void* W,
                              const float* radial_w, float* out, float* z_save, int32_t* perm, int32_t* offsets,
                              void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (p->feat_dtype != TDN_F32) return TDN_ERR_BAD_DTYPE;
  if (p->L < 2 || p->L > 4 || p->R > kChunkR) return TDN_ERR_BAD_SHAPE;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C;
  if (!A || !A2 || !B || !D || !W || !radial_w || !offsets || !workspace) return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const FwdLayout lay = fwd_layout(*p);
  if (workspace_bytes < lay.total) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, p->edges_sorted, stream);
    if (st != TDN_OK) return st;
  }
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  {
    Timed t("sort", stream);
    if (p->edges_sorted || E == 0)
      TDN_HIP(tdn::launch_offsets_presorted(N, E, dst, perm, offsets, stream));
    else
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), dst, 1, perm, offsets, ws + lay.sort, stream));
  }
  if (N == 0) return TDN_OK;
  float* Z = z_save ? z_save : reinterpret_cast<float*>(ws + lay.z);
  void* xt = ws + lay.xt;
  {
    Timed t("feature_layout", stream);
    TDN_HIP(edge_features(*p, x, true, xt, stream));
  }
  {
    Timed t("cp_edge_fwd_t3", stream);
    tdn::EdgeArgs a = edge_args(*p, offsets, perm, src, dst, edge_vec, A, D, B, radial_w, xt, Z,
                                reinterpret_cast<float*>(ws + lay.part), true);
    a.KF2 = A2;
    TDN_HIP(tdn::launch_cp_edge_t3(a, stream));
  }
  {
    Timed t("node_gemm", stream);
    TDN_HIP(tdn::launch_node_gemm(N * d, C, Z, W, false, 0, out, ws + lay.wp, stream));
  }
  return TDN_OK;
}

tdn_status tdn_ps_linear_workspace_size(int32_t C, int32_t w_dtype, size_t* bytes) {
  if (!bytes) return TDN_ERR_NULL_POINTER;
  if (w_dtype != TDN_F32 && w_dtype != TDN_BF16) return TDN_ERR_BAD_DTYPE;
  if (C < 16 || C > 256 || C % 16 != 0) return TDN_ERR_BAD_SHAPE;
  *bytes = w_dtype == TDN_F32 ? tdn::node_gemm_ws_bytes(C) : 0;
  return TDN_OK;
}

tdn_status tdn_ps_linear(int32_t n_nodes, int32_t L, int32_t C, const float* x, const void* W, int32_t w_dtype,
                         float* y, void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (w_dtype != TDN_F32 && w_dtype != TDN_BF16) return TDN_ERR_BAD_DTYPE;
  if (n_nodes < 0 || L < 0 || L > 6 || C < 16 || C > 256 || C % 16 != 0) return TDN_ERR_BAD_SHAPE;
  if (int64_t(n_nodes) * dim_of(L) >= (int64_t(1) << 31) - 1) return TDN_ERR_BAD_SHAPE;
  const bool f32 = w_dtype == TDN_F32;
  if (!W || (f32 && !workspace)) return TDN_ERR_NULL_POINTER;
  if (n_nodes > 0 && (!x || !y)) return TDN_ERR_NULL_POINTER;
  if (f32 && workspace_bytes < tdn::node_gemm_ws_bytes(C)) return TDN_ERR_WORKSPACE_TOO_SMALL;
  const tdn_status st = check_device();
  if (st != TDN_OK) return st;
  if (n_nodes == 0) return TDN_OK;
  Timed t("node_gemm", stream);
  TDN_HIP(tdn::launch_node_gemm(n_nodes * dim_of(L), C, x, W, !f32, 0, y, workspace, stream));
  return TDN_OK;
}

tdn_status tdn_dense_tp_forward(const tdn_problem* p, const void* x, const float* edge_vec,
                                const int32_t* edge_index, const int32_t* cg_row, const int32_t* cg_col,
                                const float* cg_val, int32_t cg_nnz, const float* path_w, const void* W, float* out,
                                float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                                size_t workspace_bytes, hipStream_t stream) {
  tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (p->feat_dtype != TDN_F32) return TDN_ERR_BAD_DTYPE;
  if (p->R != tdn::dense_path_count(p->L) || cg_nnz < 0) return TDN_ERR_BAD_SHAPE;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C;
  if (!cg_row || (cg_nnz > 0 && (!cg_col || !cg_val)) || !path_w || !W || !offsets || !workspace)
    return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const FwdLayout lay = fwd_layout(*p);
  if (workspace_bytes < lay.total) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, p->edges_sorted, stream);
    if (st != TDN_OK) return st;
  }
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  {
    Timed t("sort", stream);
    if (p->edges_sorted || E == 0)
      TDN_HIP(tdn::launch_offsets_presorted(N, E, dst, perm, offsets, stream));
    else
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), dst, 1, perm, offsets, ws + lay.sort, stream));
  }
  if (N == 0) return TDN_OK;
  float* Z = z_save ? z_save : reinterpret_cast<float*>(ws + lay.z);
  void* xt = ws + lay.xt;
  {
    Timed t("feature_layout", stream);
    TDN_HIP(tdn::launch_feature_layout(N, d, C, x, true, 2, xt, row_scales(*p, xt), stream));
  }
  {
    Timed t("dense_edge_fwd", stream);
    tdn::DenseArgs a{};
    a.N = N;
    a.E = E;
    a.L = p->L;
    a.d = d;
    a.C = C;
    a.n_radial = p->n_radial;
    a.n_path = p->R;
    a.cg_nnz = cg_nnz;
    a.sigma = p->r_cut / float(p->n_radial - 1);
    a.offsets = offsets;
    a.perm = perm;
    a.src = src;
    a.edge_vec = edge_vec;
    a.cg_row = cg_row;
    a.cg_col = cg_col;
    a.cg_val = cg_val;
    a.path_w = path_w;
    a.feat = xt;
    a.row_scale = row_scales(*p, xt);
    a.out = Z;
    TDN_HIP(tdn::launch_dense_edge(a, stream));
  }
  {
    Timed t("node_gemm", stream);
    TDN_HIP(tdn::launch_node_gemm(N * d, C, Z, W, false, 0, out, ws + lay.wp, stream));
  }
  return TDN_OK;
}

namespace {
size_t unshared_zp_bytes(const tdn_problem& p) {
  return size_t(p.n_nodes) * tdn::path_rows(p.L).n_rows * p.C * 4;
}
tdn_status check_unshared(const tdn_problem* p) {
  const tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  if (p->feat_dtype != TDN_F32) return TDN_ERR_BAD_DTYPE;
  if (p->R != tdn::dense_path_count(p->L) || p->C > 128) return TDN_ERR_BAD_SHAPE;
  return TDN_OK;
}
}  // namespace

tdn_status tdn_dense_tp_unshared_workspace_size(const tdn_problem* p, size_t* bytes) {
  const tdn_status st = check_unshared(p);
  if (st != TDN_OK) return st;
  if (!bytes) return TDN_ERR_NULL_POINTER;
  *bytes = fwd_layout(*p).total + al(unshared_zp_bytes(*p));
  return TDN_OK;
}

tdn_status tdn_dense_tp_forward_unshared(const tdn_problem* p, const void* x, const float* edge_vec,
                                         const int32_t* edge_index, const int32_t* cg_row, const int32_t* cg_col,
                                         const float* cg_val, int32_t cg_nnz, const float* path_w,
                                         const float* W_paths, float* out, int32_t* perm, int32_t* offsets,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream) {
  tdn_status st = check_unshared(p);
  if (st != TDN_OK) return st;
  if (cg_nnz < 0) return TDN_ERR_BAD_SHAPE;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C;
  if (!cg_row || (cg_nnz > 0 && (!cg_col || !cg_val)) || !path_w || !W_paths || !offsets || !workspace)
    return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const FwdLayout lay = fwd_layout(*p);
  if (workspace_bytes < lay.total + al(unshared_zp_bytes(*p))) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, p->edges_sorted, stream);
    if (st != TDN_OK) return st;
  }
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  {
    Timed t("sort", stream);
    if (p->edges_sorted || E == 0)
      TDN_HIP(tdn::launch_offsets_presorted(N, E, dst, perm, offsets, stream));
    else
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), dst, 1, perm, offsets, ws + lay.sort, stream));
  }
  if (N == 0) return TDN_OK;
  float* zp = reinterpret_cast<float*>(ws + lay.total);
  void* xt = ws + lay.xt;
  {
    Timed t("feature_layout", stream);
    TDN_HIP(tdn::launch_feature_layout(N, d, C, x, true, 2, xt, row_scales(*p, xt), stream));
  }
  {
    Timed t("dense_edge_unshared", stream);
    tdn::DenseArgs a{};
    a.N = N;
    a.E = E;
    a.L = p->L;
    a.d = d;
    a.C = C;
    a.n_radial = p->n_radial;
    a.n_path = p->R;
    a.cg_nnz = cg_nnz;
    a.sigma = p->r_cut / float(p->n_radial - 1);
    a.offsets = offsets;
    a.perm = perm;
    a.src = src;
    a.edge_vec = edge_vec;
    a.cg_row = cg_row;
    a.cg_col = cg_col;
    a.cg_val = cg_val;
    a.path_w = path_w;
    a.feat = xt;
    a.row_scale = row_scales(*p, xt);
    TDN_HIP(tdn::launch_dense_edge_unshared(a, zp, stream));
  }
  {
    Timed t("path_gemm", stream);
    TDN_HIP(tdn::launch_path_gemm(N, p->L, C, zp, W_paths, out, stream));
  }
  return TDN_OK;
}

tdn_status tdn_cp_tp_backward(const tdn_problem* p, const void* x, const float* edge_vec, const int32_t* edge_index,
                              const float* A, const float* B, const float* D, const void* W, const float* radial_w,
                              const int32_t* perm, const int32_t* offsets, const float* z_save,
                              const float* grad_out, float* grad_x, float* grad_W, float* grad_edge_vec,
                              float* grad_radial_w, void* workspace, size_t workspace_bytes,
                              hipStream_t stream) {
  tdn_status st = check_problem(p);
  if (st != TDN_OK) return st;
  const int N = p->n_nodes, E = p->n_edges, d = dim_of(p->L), C = p->C;
  if (!A || !B || !D || !W || !radial_w || !offsets || !workspace) return TDN_ERR_NULL_POINTER;
  if (N > 0 && (!x || !grad_out)) return TDN_ERR_NULL_POINTER;
  if (E > 0 && (!edge_vec || !edge_index || !perm)) return TDN_ERR_NULL_POINTER;
  const BwdLayout lay = bwd_layout(*p);
  if (workspace_bytes < lay.total) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  char* ws = static_cast<char*>(workspace);
  if (p->validate) {
    st = run_validation(*p, edge_index, edge_vec, ws, lay.flags, 0, stream);
    if (st != TDN_OK) return st;
  }
  const bool bf16 = p->feat_dtype == TDN_BF16;
  const int32_t* src = edge_index;
  const int32_t* dst = E > 0 ? edge_index + E : nullptr;
  if (N == 0 || E == 0) {
    if (grad_radial_w) TDN_HIP(tdn::launch_zero(grad_radial_w, size_t(p->n_radial) * p->R * 4, stream));
  }
  if (N == 0) {
    if (grad_W) TDN_HIP(tdn::launch_zero(grad_W, size_t(C) * C * 4, stream));
    return TDN_OK;
  }
  float* Gz = reinterpret_cast<float*>(ws + lay.gz);
  {
    Timed t("node_gemm", stream);
    TDN_HIP(tdn::launch_node_gemm(N * d, C, grad_out, W, bf16, 1, Gz, ws + lay.wp, stream));
  }
  if (grad_W) {
    const float* Z = z_save;
    if (!Z) {
      float* Zw = reinterpret_cast<float*>(ws + lay.z);
      TDN_HIP(forward_edge_pass(*p, offsets, perm, src, dst, edge_vec, A, B, D, radial_w, x, ws + lay.xt,
                                reinterpret_cast<float*>(ws + lay.part), Zw, reinterpret_cast<float*>(ws + lay.fsl),
                                reinterpret_cast<float*>(ws + lay.gtmp), stream));
      Z = Zw;
    }
    Timed t("gram", stream);
    TDN_HIP(tdn::launch_gram(N * d, C, Z, grad_out, bf16, reinterpret_cast<float*>(ws + lay.parts), grad_W, stream));
  }
  const int nch = rank_chunks(p->R);
  float* fsl = reinterpret_cast<float*>(ws + lay.fsl);
  float *sA = fsl, *sB = fsl + size_t(d) * kChunkR, *sD = fsl + size_t(2 * d) * kChunkR;
  float* sW = fsl + size_t(3 * d) * kChunkR;
  float* gtmp = reinterpret_cast<float*>(ws + lay.gtmp);
  // the factor and radial-weight columns of rank chunk c (the inputs
  // themselves when the problem is one chunk)
  auto chunk_inputs = [&](int c, int* r0, int* n, const float** cA, const float** cB, const float** cD,
                          const float** cW) -> hipError_t {
    chunk_range(p->R, c, nch, r0, n);
    if (nch == 1) {
      *cA = A, *cB = B, *cD = D, *cW = radial_w;
      return hipSuccess;
    }
    hipError_t e = tdn::launch_slice_cols(d, p->R, *r0, *n, A, sA, stream);
    if (e == hipSuccess) e = tdn::launch_slice_cols(d, p->R, *r0, *n, B, sB, stream);
    if (e == hipSuccess) e = tdn::launch_slice_cols(d, p->R, *r0, *n, D, sD, stream);
    if (e == hipSuccess) e = tdn::launch_slice_cols(p->n_radial, p->R, *r0, *n, radial_w, sW, stream);
    *cA = sA, *cB = sB, *cD = sD, *cW = sW;
    return e;
  };
  if ((grad_edge_vec || grad_radial_w) && E > 0) {
    // dL/dr_e and dL/drho are sums over ranks: per rank chunk, the edge
    // gradients go to the output (first chunk) or to gtmp and are added in
    // chunk order; the radial-weight gradient of the chunk fills its columns
    float* gv_out = grad_edge_vec ? grad_edge_vec : reinterpret_cast<float*>(ws + lay.gv);
    // the split form takes Gz in the layout of xc (independent of the rank chunk)
    const bool split = tdn::bwd_dst_split(p->L, C, bf16) && tdn::bwd_dst_plan(p->L, chunk_problem(*p, 0).R, C,
                                                                               p->n_radial, bf16, E).n_range > 0;
    float* gzscale = reinterpret_cast<float*>(ws + lay.gzc + al(xc_bytes(*p)));
    if (split) {
      Timed t("channel_layout", stream);
      TDN_HIP(tdn::launch_direct_layout(N, d, C, tdn::bwd_dst_cpad(C, bf16), Gz, true, feature_parts(*p),
                                        ws + lay.gzc, bf16 ? nullptr : gzscale, false, stream));
    }
    for (int c = 0; c < nch; ++c) {
      int r0 = 0, n = 0;
      const float *cA, *cB, *cD, *cW;
      TDN_HIP(chunk_inputs(c, &r0, &n, &cA, &cB, &cD, &cW));
      tdn::BwdDstArgs a{};
      a.n_seg = N;
      a.E = E;
      a.L = p->L;
      a.d = d;
      a.C = C;
      a.R = n;
      a.n_radial = p->n_radial;
      a.sigma = p->r_cut / float(p->n_radial - 1);
      a.offsets = offsets;
      a.perm = perm;
      a.src = src;
      a.edge_vec = edge_vec;
      a.A = cA;
      a.Bf = cB;
      a.D = cD;
      a.radial_w = cW;
      a.x = x;
      a.Gz = Gz;
      a.grad_vec = c == 0 ? gv_out : gtmp;
      a.drho = grad_radial_w ? reinterpret_cast<float*>(ws + lay.drho) : nullptr;
      a.dst = dst;
      const tdn::EdgePlan dp = tdn::bwd_dst_plan(p->L, n, C, p->n_radial, bf16, E);
      a.n_range = dp.n_range;
      a.pieces_per_block = dp.per_block;
      if (a.n_range > 0) {
        // x in parts (fp16 with row scales for fp32 problems, bf16), blocked as
        // MFMA operands for the contraction over channels (the region is free
        // until the grad_x pass lays out Gz there)
        float* xscale = reinterpret_cast<float*>(ws + lay.xt + al(xc_bytes(*p)));
        Timed t("channel_layout", stream);
        TDN_HIP(tdn::launch_direct_layout(N, d, C, tdn::bwd_dst_cpad(C, bf16), x, !bf16, feature_parts(*p),
                                          ws + lay.xt, bf16 ? nullptr : xscale, false, stream));
        a.xc = ws + lay.xt;
        a.x_scale = bf16 ? nullptr : xscale;
        // the range kernel sums the radial-weight gradient per workgroup
        a.drho = nullptr;
        a.wrad_part = grad_radial_w ? reinterpret_cast<float*>(ws + lay.wrad_part) : nullptr;
        if (split) {
          a.gzc = ws + lay.gzc;
          a.gz_scale = bf16 ? nullptr : gzscale;
          a.dg = reinterpret_cast<float*>(ws + lay.drho);
        }
      } else if (d > 32) {
        // x in the direct kernel's operand blocks, channels in its accumulator
        // order
        float* xscale = reinterpret_cast<float*>(ws + lay.xt + al(xd_bytes(*p)));
        Timed t("channel_layout", stream);
        TDN_HIP(tdn::launch_direct_layout(N, d, C, tdn::bwd_direct_cpad(C), x, !bf16, feature_parts(*p),
                                          ws + lay.xt, bf16 ? nullptr : xscale, true, stream));
        a.xc = ws + lay.xt;
        a.x_scale = bf16 ? nullptr : xscale;
        a.bt = reinterpret_cast<float*>(ws + lay.bt);
      }
      {
        Timed t("cp_bwd_dst", stream);
        TDN_HIP(tdn::launch_bwd_dst(a, bf16, stream));
        if (c > 0) TDN_HIP(tdn::launch_accumulate(size_t(E) * 3, gtmp, gv_out, stream));
      }
      if (grad_radial_w) {
        Timed t("radial_grad", stream);
        float* gr = nch == 1 ? grad_radial_w : reinterpret_cast<float*>(ws + lay.grtmp);
        if (a.n_range > 0)
          TDN_HIP(tdn::launch_sum_parts(a.n_range / a.pieces_per_block, p->n_radial * n, a.wrad_part, gr, stream));
        else
          TDN_HIP(tdn::launch_radial_grad(E, n, p->n_radial, a.sigma, edge_vec, a.drho,
                                          reinterpret_cast<float*>(ws + lay.wrad_part), gr, stream));
        if (nch > 1) TDN_HIP(tdn::launch_scatter_cols(p->n_radial, p->R, r0, n, gr, grad_radial_w, stream));
      }
    }
  }
  if (grad_x) {
    int32_t* perm_src = reinterpret_cast<int32_t*>(ws + lay.perm_src);
    int32_t* off_src = reinterpret_cast<int32_t*>(ws + lay.off_src);
    {
      Timed t("sort", stream);
      TDN_HIP(tdn::launch_sort(tdn::sort_plan(N, E), src, 1, perm_src, off_src, ws + lay.sort, stream));
    }
    // bf16 problems run the grad_x pass on bf16 MFMA too (Gz rounded to
    // bf16); fp32 problems on the fp16 two-part split of Gz
    {
      Timed t("feature_layout", stream);
      TDN_HIP(edge_features(*p, Gz, true, ws + lay.xt, stream));
    }
    Timed t("cp_edge_bwd_src", stream);
    TDN_HIP(edge_pass_ranks(*p, off_src, perm_src, dst, src, edge_vec, D, A, B, radial_w, ws + lay.xt, grad_x,
                            reinterpret_cast<float*>(ws + lay.part), fsl, gtmp, stream));
  }
  return TDN_OK;
}

tdn_status tdn_sort_workspace_size(int32_t n_keys, int32_t E, size_t* bytes) {
  if (!bytes) return TDN_ERR_NULL_POINTER;
  if (n_keys < 0 || E < 0 || (E > 0 && n_keys == 0)) return TDN_ERR_BAD_SHAPE;
  *bytes = tdn::sort_plan(n_keys, E).bytes + 256;
  return TDN_OK;
}

tdn_status tdn_sort_by_key(int32_t n_keys, int32_t E, const int32_t* keys, int32_t* perm, int32_t* offsets,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (n_keys < 0 || E < 0 || (E > 0 && n_keys == 0)) return TDN_ERR_BAD_SHAPE;
  if (!offsets || !workspace || (E > 0 && (!keys || !perm))) return TDN_ERR_NULL_POINTER;
  const tdn::SortPlan plan = tdn::sort_plan(n_keys, E);
  if (workspace_bytes < plan.bytes + 256) return TDN_ERR_WORKSPACE_TOO_SMALL;
  tdn_status st = check_device();
  if (st != TDN_OK) return st;
  Timed t("sort", stream);
  TDN_HIP(tdn::launch_sort(plan, keys, 1, perm, offsets, workspace, stream));
  return TDN_OK;
}

namespace {
tdn_status check_graph_problem(const tdn_graph_problem* g) {
  if (!g) return TDN_ERR_NULL_POINTER;
  if (g->n_nodes < 0 || g->n_nodes >= (1 << 26) || g->n_graphs < 0 || g->max_neighbors < 0)
    return TDN_ERR_BAD_SHAPE;
  if (g->n_nodes > 0 && g->n_graphs == 0) return TDN_ERR_BAD_SHAPE;
  if (g->n_graphs > (1 << 26)) return TDN_ERR_BAD_SHAPE;
  if (!(g->r_cut > 0.f) || !std::isfinite(g->r_cut)) return TDN_ERR_BAD_SHAPE;
  for (int k = 0; k < 3; ++k)
    if (g->periodic[k] != 0 && g->periodic[k] != 1) return TDN_ERR_BAD_SHAPE;
  return TDN_OK;
}
}  // namespace

tdn_status tdn_radius_graph_workspace_size(const tdn_graph_problem* g, size_t* bytes) {
  const tdn_status st = check_graph_problem(g);
  if (st != TDN_OK) return st;
  if (!bytes) return TDN_ERR_NULL_POINTER;
  *bytes = tdn::radius_graph_layout(g->n_nodes, g->n_graphs).total;
  return TDN_OK;
}

tdn_status tdn_radius_graph(const tdn_graph_problem* g, const float* pos, const int32_t* graph_ptr,
                            const float* cell, int64_t edge_capacity, int32_t* edge_index, float* edge_vec,
                            int32_t* edge_image, int32_t* offsets, int64_t* n_edges, void* workspace,
                            size_t workspace_bytes, hipStream_t stream) {
  tdn_status st = check_graph_problem(g);
  if (st != TDN_OK) return st;
  if (!n_edges || !graph_ptr || !workspace || (g->n_nodes > 0 && !pos)) return TDN_ERR_NULL_POINTER;
  const bool periodic = g->periodic[0] || g->periodic[1] || g->periodic[2];
  if (periodic && g->n_graphs > 0 && !cell) return TDN_ERR_NULL_POINTER;
  if (edge_capacity < 0) return TDN_ERR_BAD_SHAPE;
  if (edge_capacity > 0 && (!edge_index || !edge_vec)) return TDN_ERR_NULL_POINTER;
  const tdn::RadiusGraphLayout lay = tdn::radius_graph_layout(g->n_nodes, g->n_graphs);
  if (workspace_bytes < lay.total) return TDN_ERR_WORKSPACE_TOO_SMALL;
  st = check_device();
  if (st != TDN_OK) return st;
  tdn::RadiusGraphArgs a{};
  a.N = g->n_nodes;
  a.G = g->n_graphs;
  a.r_cut = g->r_cut;
  a.max_neighbors = g->max_neighbors;
  for (int k = 0; k < 3; ++k) a.periodic[k] = g->periodic[k];
  a.pos = pos;
  a.graph_ptr = graph_ptr;
  a.cell = cell;
  char* ws = static_cast<char*>(workspace);
  Timed t("radius_graph", stream);
  TDN_HIP(tdn::launch_radius_count(a, ws, stream));
  int32_t flags[5] = {0, 0, 0, 0, 0}, total = 0;
  TDN_HIP(hipMemcpyAsync(flags, ws + lay.flags, sizeof(flags), hipMemcpyDeviceToHost, stream));
  TDN_HIP(hipMemcpyAsync(&total, ws + lay.offs + size_t(a.N) * 4, 4, hipMemcpyDeviceToHost, stream));
  TDN_HIP(hipStreamSynchronize(stream));
  if (flags[0] || flags[1]) return TDN_ERR_BAD_GEOMETRY;
  if (flags[2]) return TDN_ERR_NEIGHBOUR_LIMIT;
  *n_edges = total;
  if (offsets)
    TDN_HIP(hipMemcpyAsync(offsets, ws + lay.offs, (size_t(a.N) + 1) * 4, hipMemcpyDeviceToDevice, stream));
  if (int64_t(total) > edge_capacity) return TDN_ERR_EDGE_CAPACITY;
  if (total > 0)
    TDN_HIP(tdn::launch_radius_emit(a, ws, flags[4], edge_index, edge_vec, edge_image, stream));
  return TDN_OK;
}

tdn_status tdn_spherical_harmonics(int32_t L, int32_t E, const float* edge_vec, float* Y, float* dY,
                                   hipStream_t stream) {
  if (L < 0 || L > 6 || E < 0) return TDN_ERR_BAD_SHAPE;
  if (E > 0 && (!edge_vec || !Y)) return TDN_ERR_NULL_POINTER;
  tdn_status st = check_device();
  if (st != TDN_OK) return st;
  TDN_HIP(tdn::launch_sh(L, E, edge_vec, Y, dY, stream));
  return TDN_OK;
}

tdn_status tdn_timer_enable(int32_t enable) {
  Timer& t = timer();
  std::lock_guard<std::mutex> lk(t.mu);
  t.on = enable != 0;
  return TDN_OK;
}

tdn_status tdn_timer_read(const char* kernel, double* total_ms, int32_t* launches, int32_t reset) {
  if (!kernel || !total_ms || !launches) return TDN_ERR_NULL_POINTER;
  Timer& t = timer();
  std::lock_guard<std::mutex> lk(t.mu);
  auto& pend = t.pending[kernel];
  auto& acc = t.done[kernel];
  for (auto& ev : pend) {
    TDN_HIP(hipEventSynchronize(ev.second));
    float ms = 0.f;
    TDN_HIP(hipEventElapsedTime(&ms, ev.first, ev.second));
    acc.first += ms;
    acc.second += 1;
    hipEventDestroy(ev.first);
    hipEventDestroy(ev.second);
  }
  pend.clear();
  *total_ms = acc.first;
  *launches = acc.second;
  if (reset) acc = {0.0, 0};
  return TDN_OK;
}

}  // extern "C"

namespace tdn {

tdn_status record_hip_error(hipError_t e) { return hip_fail(e); }

tdn_status require_gfx950() { return check_device(); }

tdn_status forward_untimed(const tdn_problem* p, const void* x, const float* edge_vec, const int32_t* edge_index,
                           const float* A, const float* B, const float* D, const void* W, const float* radial_w,
                           float* out, float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  g_untimed = true;
  const tdn_status st = forward_impl(p, x, edge_vec, edge_index, A, B, D, W, radial_w, out, z_save, perm, offsets,
                                     workspace, workspace_bytes, stream, false);
  g_untimed = false;
  return st;
}

}  // namespace tdn
