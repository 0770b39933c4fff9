// Internal launch interface between the C ABI (api.cpp) and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace tdn {

// ---------------------------------------------------------------- sorting
// Stable LSD radix sort of int keys in [0, n_keys) with 8-bit digits.
struct SortPlan {
  int n_keys, E, passes, n_blocks;
  size_t bytes;  // workspace bytes
};
SortPlan sort_plan(int n_keys, int E);
// keys: [E] input; perm [E]; offsets [n_keys+1]; ws from sort_plan.
hipError_t launch_sort(const SortPlan& plan, const int32_t* keys, int key_stride, int32_t* perm,
                       int32_t* offsets, void* ws, hipStream_t s);
// offsets from keys already sorted (non-decreasing); perm = identity.
hipError_t launch_offsets_presorted(int n_keys, int E, const int32_t* sorted_keys, int32_t* perm,
                                    int32_t* offsets, hipStream_t s);
// Exclusive prefix sum of n ints in place (one workgroup).
hipError_t launch_scan_exclusive(int32_t* a, int n, hipStream_t s);
// Device-side validation; flags (3 ints, cleared by this call): [0] index
// range, [1] dst order, [2] degenerate edge vector.
hipError_t launch_validate(int N, int E, const int32_t* edge_index, const float* edge_vec, int check_sorted,
                           int32_t* flags, hipStream_t s);

// ---------------------------------------------------------------- edge kernel
// One Khatri-Rao contraction pass over segments of a sorted edge list:
//   H_seg = sum_{e in seg} diag(g_e) KF^T feat[gather[e]]    ([R, C])
//   out[seg] = EF H_seg                                       ([d, C])
// forward:        KF = A, EF = D, feat = x,  gather = src, key = dst
// grad_x pass:    KF = D, EF = A, feat = Gz, gather = dst, key = src
// The pass splits the sorted edges into n_range equal ranges, several per
// workgroup; segments spanning ranges are summed from `partial`
// ([n_range, 2, d, C] floats of workspace).
struct EdgeArgs {
  int n_seg, E, L, d, C, R, n_radial;
  float sigma;               // r_cut / (n_radial - 1)
  const int32_t* offsets;    // [n_seg + 1]
  const int32_t* perm;       // [E] sorted slot -> edge id
  const int32_t* gather;     // [E] by edge id: row of feat to gather
  const int32_t* key;        // [E] by edge id: segment of the edge
  const float* edge_vec;     // [E, 3] by edge id
  const float* KF;           // [d, R]
  const float* EF;           // [d, R]
  const float* Bf;           // [d, R]
  const float* radial_w;     // [n_radial, R]
  const float* KF2;          // [d, R] second node factor of the three-input product (launch_cp_edge_t3 only)
  const void* feat;          // parts = 2: launch_feature_layout_packed's words; parts = 1: the bf16 blocks
                             // of launch_feature_layout
  float* out;                // [n_seg, d, C]
  int n_range;               // edge ranges (EdgePlan::n_range)
  int pieces_per_block;      // ranges per workgroup (EdgePlan::per_block)
  float* partial;            // [n_range, 2, d, C] workspace
  void* ef_ops;              // workspace of edge_ef_bytes(d, R): EF in the epilogue's operand blocks
                             // and its scale (written by launch_cp_edge)
  float* ef_scale;           // inside ef_ops: 2^e of EF's fp16 parts (parts = 2)
  int parts;                 // 16-bit parts per feature in feat (2: fp32 features as fp16 hi + lo, 1: bf16)
  const float* row_scale;    // [n_feat_rows] 2^e of each feat row (parts = 2), from launch_feature_layout
  // attention (launch_cp_edge_att): the weights [E, n_heads] by sorted position
  const float* alpha;
  int n_heads;
  // measurement ablations only (launch_cp_edge_ablation):
  void* fa_global;           // factors from global memory: per workgroup a copy of its packed factor blocks
  const float* y_table;      // harmonics table: [E, d] Y of each edge by edge id (launch_sh)
};
// Edge ranges of the pass for this problem on the current device:
// n_range = per_block x the number of workgroups the device holds at once
// over the channel groups (capped at E; 0 when E = 0).  Workgroup b takes
// ranges b, b + n_range / per_block, ...
struct EdgePlan {
  int n_range, per_block;
};
EdgePlan edge_plan(int L, int R, int C, int n_radial, bool bf16, int E, bool t3 = false);
// Features for the edge pass: x [N, d, C] -> 32x32x16 MFMA operand blocks
// xs [N, ceil(C/32), parts, edge_kpad(d)/16, 2, 32, 8] of 16-bit values,
// element [n][ct][s][b][h][c][i] = part s of x[n][16b + 8h + i][32ct + c],
// zero padded in k and c (EdgeArgs::feat = xs).  parts = 2 (fp32 features):
// fp16 hi and lo of x[n] 2^-e_n with x[n] 2^-e_n = hi + lo to 2^-22, e_n
// putting the row's largest |x| in [2^13, 2^14), and row_scale[n] = 2^e_n;
// parts = 1: bf16 features (an fp32 input is rounded to bf16; row_scale is
// not used).  edge_kpad(d) = 32 for d <= 32, else 64.
int edge_kpad(int d);
hipError_t launch_feature_layout(int N, int d, int C, const void* x, bool x_is_f32, int parts, void* xs,
                                 float* row_scale, hipStream_t s);
// Packed split operands of the edge pass for fp32 features (the layout
// launch_cp_edge reads when parts = 2).  With n = pk_rows(d) = ceil(d / 2),
// lane half h of a 32x32x16 MFMA owns degree rows h n .. h n + n - 1 and gives
// each of them three K slots: (x hi, factor hi), (x lo, factor hi),
// (x hi, factor lo), grouped as slots [0, n), [n, 2n), [2n, 3n) of the
// lane's 8 pk_blocks(d) slots (the rest pair with zero factor values), so
// the three part products of the fp32-level contraction are one K-reduction
// of pk_blocks(d) steps.  x'[node] = x[node] 2^-e_node as in
// launch_feature_layout (row_scale[node] = 2^e_node).  Lane (h, c) of channel
// tile ct stores n words, word j = fp16 values 2j, 2j + 1 of the sequence
// (hi of rows h n .., then lo of rows h n ..); per node and tile the words
// are [n / 4][64 lanes][4] then [64 lanes][n % 4]: 256 n bytes.  The slots
// [2n, 3n) reuse the first words, so each value is loaded once.
__host__ __device__ constexpr int pk_rows(int d) { return (d + 1) / 2; }
__host__ __device__ constexpr int pk_blocks(int d) { return (3 * pk_rows(d) + 7) / 8; }
hipError_t launch_feature_layout_packed(int N, int d, int C, const float* x, void* xp, float* row_scale,
                                        hipStream_t s);
// Features for the backward's destination kernels, blocked for contractions
// over channels: xd [N, parts, Cp / 16, 2, d, 8] of 16-bit values, element
// [n][p][s][h][k][i] = part p of x[n][k][c(s, h, i)] with c = 16 s + 8 h + i,
// or with perm_channels c = 16 s + 8 (i / 4) + 4 h + i % 4 (the direct
// kernel's accumulator order); zero from channel C, Cp a multiple of 16.
// parts = 2: fp16 hi and lo of x[n] 2^-e_n and row_scale[n] = 2^e_n as for
// the edge pass; parts = 1: bf16.
hipError_t launch_direct_layout(int N, int d, int C, int Cp, const void* x, bool x_is_f32, int parts, void* xd,
                                float* row_scale, bool perm_channels, hipStream_t s);
// parts = 2: fp32 features (fp16 two-part split), parts = 1: bf16 features
hipError_t launch_cp_edge(const EdgeArgs& a, hipStream_t s);
// Measurement ablation of the segmented sum (fp32 features, 2 <= L <= 4): the
// same contraction with every edge its own segment, the output factor applied
// per edge and Z accumulated into `out` (zeroed first) with float atomics;
// nondeterministic in the order of the additions.
hipError_t launch_cp_edge_atomic(const EdgeArgs& a, hipStream_t s);
// The attention block's edge pass (fp32 features, 1 <= L <= 4, one rank
// chunk): launch_cp_edge with every edge's message weighted per head by
// a.alpha[sorted position][head] before the segment sum (a.n_heads heads of
// C / n_heads channels each, a multiple of 32, n_heads <= 8).
hipError_t launch_cp_edge_att(const EdgeArgs& a, hipStream_t s);
// Its weights.  launch_att_node: per node the hidden projections of the
// degree-0 row, Pt[n] = x[n][0] W1[0 .. C) and Ps[n] = x[n][0] W1[C .. 2C)
// ([N, F] each; W1 [2C + n_radial, F] row-major).  launch_att_alpha: per
// destination (one wave), for its edges in sorted order the logits
// a_e = LeakyReLU(Pt[t] + Ps[s_e] + phi_e W1[2C ..], 0.2) w2 (w2 [F, H]), then
// the softmax over the destination's edges per head into alpha_sorted
// [E, H] (sorted position) and, if not NULL, alpha_eid [E, H] (edge id).
// F <= 64, H <= 8.
hipError_t launch_att_node(int N, int d, int C, int F, const float* x, const float* W1, float* Pt, float* Ps,
                           hipStream_t s);
hipError_t launch_att_alpha(int N, int C, int F, int H, int n_radial, float sigma, const int32_t* offsets,
                            const int32_t* perm, const int32_t* src, const float* edge_vec, const float* Pt,
                            const float* Ps, const float* W1, const float* w2, float* alpha_sorted,
                            float* alpha_eid, hipStream_t s);
// Measurement ablations of the edge pass (fp32 features, 2 <= L <= 4, one
// rank chunk), each with one hot-path choice replaced:
//   kAblFactorsGlobal: the packed factor blocks read in the edge loop from a
//     per-workgroup copy in global memory (a.fa_global, edge_abl_fa_bytes)
//     instead of registers or LDS;
//   kAblYTable: the harmonics read from a precomputed table (a.y_table)
//     instead of evaluated in the kernel;
//   kAblValu: the contraction, the segment sum and D on the vector ALUs in
//     fp32 (one workgroup per destination, R <= 128, C <= 128), reading x
//     itself (x_f32 [N, d, C]) instead of the packed split words.
// The first two keep everything else of launch_cp_edge.
constexpr int kAblFactorsGlobal = 1, kAblYTable = 2, kAblValu = 3;
hipError_t launch_cp_edge_ablation(const EdgeArgs& a, int variant, const float* x_f32, hipStream_t s);
size_t edge_abl_fa_bytes(int L, int R, int C, int n_range, int pieces_per_block);
// kAblValu's kernel: out[t] = D sum_e diag(g_e) A^T x[src_e] per destination t
// in fp32 FMA (L <= 4, R <= 128, C <= 128), zero rows for nodes without
// edges; a.KF = A, a.EF = D, a.Bf, a.radial_w, a.offsets, a.perm, a.gather,
// a.edge_vec as for launch_cp_edge.
hipError_t launch_cp_edge_valu(const EdgeArgs& a, const float* x, hipStream_t s);
// The three-input product (App. A, N = 3: source features, edge harmonics,
// destination features): as launch_cp_edge, with each segment's sum
// multiplied by V_t = KF2^T x[t] (t = the segment's node, a row of feat)
// before EF is applied.  fp32 features, 2 <= L <= 4; the plan must come from
// edge_plan(..., t3 = true).
hipError_t launch_cp_edge_t3(const EdgeArgs& a, hipStream_t s);

// The exact CG tensor product over the sorted edges (the comparator of the CP
// edge pass): out[n] = sum over edges e into n of K_e x[src_e] with
// K_e[k][i] = sum_j C[k; i, j] Y_e[j] rho_e[path], rho_e = phi_e path_w.
// The coefficients come as rows over (k, i) pairs, q = k d + i: entries
// cg_row[q] .. cg_row[q+1] - 1 of cg_col (j | path << 16) and cg_val.  Rows
// are clamped to [0, cg_nnz] and entries with j >= d or path >= n_path are
// skipped, so any table stays in bounds.  fp32 features only (feat in
// launch_feature_layout's blocks with parts = 2, and its row scales).
struct DenseArgs {
  int N, E, L, d, C, n_radial, n_path, cg_nnz;
  float sigma;             // r_cut / (n_radial - 1)
  const int32_t* offsets;  // [N + 1]
  const int32_t* perm;     // [E] sorted slot -> edge id
  const int32_t* src;      // [E] by edge id
  const float* edge_vec;   // [E, 3] by edge id
  const int32_t* cg_row;   // [d * d + 1]
  const int32_t* cg_col;   // [cg_nnz]
  const float* cg_val;     // [cg_nnz]
  const float* path_w;     // [n_radial, n_path]
  const void* feat;        // operand blocks of x (parts = 2)
  const float* row_scale;  // [N]
  float* out;              // [N, d, C]
};
// Paths (l1, l2, l3) of the full product up to degree L.
int dense_path_count(int L);
hipError_t launch_dense_edge(const DenseArgs& a, hipStream_t s);

// out[i] = sum over p = 0 .. n_part - 1 of partial[p][i] (i < n), in a fixed
// order (sixteen strided partial sums, then those in order; above 256 parts
// first the groups of 64 consecutive parts, each written over its first
// part, so partial is overwritten then)
hipError_t launch_sum_parts(int n_part, int n, float* partial, float* out, hipStream_t s);
// The product without path-weight sharing: every path keeps its own block of
// output rows, path p (in the order l1, then l2, then l3 ascending) owning
// rows row[p] .. row[p] + 2 l3[p], n_rows = sum over paths of 2 l3 + 1.
// first[l1 (L + 1) + l2] is the index of the path (l1, l2, |l1 - l2|).
constexpr int kMaxPaths = 176;
constexpr int kMaxDegPairs = 49;
struct PathRows {
  int n_path, n_rows;
  int l1[kMaxPaths], l2[kMaxPaths], l3[kMaxPaths];
  int row[kMaxPaths];
  int first[kMaxDegPairs];
};
PathRows path_rows(int L);
// zp[n][row][c] = the sum over edges into n of the edge's path blocks,
// zp[n][row[p] + m3] = sum_e rho_e[p] sum_{i, j} C[(l3, m3); i, j] x[s_e][i] Y_e[j]
// for the entries of path p (fp32 features, C <= 128).
hipError_t launch_dense_edge_unshared(const DenseArgs& a, float* zp, hipStream_t s);
// out[n][(l3, m3)][:] = sum over paths p with degree l3 of zp[n][row[p] + m3][:] W_paths[p]
// (W_paths [P, C, C] fp32, [in][out] per path; fp32 operands on the
// GEMM's fp32 path).
hipError_t launch_path_gemm(int N, int L, int C, const float* zp, const float* W_paths, float* out, hipStream_t s);
// Workspace bytes of EdgeArgs::ef_ops: the output factor in 32x32x16 operand
// blocks [ceil(d/32)][ceil(R/32)][2][parts][64 lanes] x 16 bytes (parts <= 2)
// (edge_ef_blocks_bytes), the node factor in the edge loop's packed blocks
// [pk_blocks(d)][ceil(R/32)][64 lanes] x 16 bytes (fp32 features), then 256
// bytes holding the two scales (EF's, then KF's).
__host__ __device__ inline size_t edge_ef_blocks_bytes(int d, int R) {
  return size_t((d + 31) / 32) * ((R + 31) / 32) * 2 * 2 * 64 * 16;
}
size_t edge_ef_bytes(int d, int R);

// ---------------------------------------------------------------- node GEMMs
// out[rows, C] = in[rows, C] @ W (transpose_w = 0) or in @ W^T (transpose_w = 1).
// fp32 W: fp16 MFMA over power-of-two scaled two-part splits of W and of each
// row of `in` (fp32-level accuracy), W's parts in ws (node_gemm_ws_bytes(C)
// bytes); w_bf16: bf16 MFMA with `in` rounded to bf16 (ws unused).  C is a
// multiple of 16.
size_t node_gemm_ws_bytes(int C);
hipError_t launch_node_gemm(int rows, int C, const float* in, const void* W, bool w_bf16, int transpose_w,
                            float* out, void* ws, hipStream_t s);
// grad_W[C, C] = sum_rows Z[row, :]^T G[row, :], split over gram_parts(rows, C)
// row chunks reduced in a fixed order.  partial: [n_part, C, C] floats of
// workspace.  bf16 = 1 rounds Z and G to bf16 for the MFMA (bf16 problems).
int gram_parts(int rows, int C);
hipError_t launch_gram(int rows, int C, const float* Z, const float* G, bool bf16, float* partial, float* grad_W,
                       hipStream_t s);

// ---------------------------------------------------------------- backward
struct BwdDstArgs {
  int n_seg, E, L, d, C, R, n_radial;
  float sigma;
  const int32_t* offsets;   // dst segments
  const int32_t* perm;
  const int32_t* src;       // [E] by edge id
  const int32_t* dst;       // [E] by edge id
  const float* edge_vec;
  const float* A;
  const float* Bf;
  const float* D;
  const float* radial_w;
  const void* x;            // [N, d, C]
  const float* Gz;          // [N, d, C] = grad_out W^T
  float* grad_vec;          // [E, 3] by edge id
  const void* xc;           // x blocked by launch_direct_layout: plain order, Cp = bwd_dst_cpad(C, bf16)
                            // (d <= 32); accumulator order, Cp = bwd_direct_cpad(C) (d > 32)
  const float* x_scale;     // fp32 problems: row_scale of launch_direct_layout
  int n_range;              // equal edge ranges (bwd_dst_plan)
  int pieces_per_block;     // ranges per workgroup
  float* drho;              // [E, R] by edge id: dL/drho_e, or nullptr (not stored); per-segment kernels
  float* bt;                // direct kernel (d > 32): workspace of (d + n_radial) R floats for B^T
                            // [R, d] and Wrad^T [R, n_radial], written by its launch
  // range kernel only:
  float* wrad_part;         // [n_range / pieces_per_block, n_radial, R]: each workgroup's share of
                            // grad_radial_w (sum them in order), or nullptr
  const void* gzc;          // Gz in the layout of xc (launch_direct_layout): selects the split form
  const float* gz_scale;    // fp32 problems: row_scale of that layout
  float* dg;                // split form: [E, R] dL/dg by sorted edge position (written, then read)
};
// Edge ranges of the destination-side kernel on the current device
// (n_range = 0 when the problem takes the per-segment kernels: d > 32 or no
// LDS fit): per_block ranges per workgroup, workgroup b taking ranges
// b, b + n_range / per_block, ...
EdgePlan bwd_dst_plan(int L, int R, int C, int n_radial, bool bf16, int E);
// whether the range kernel takes the split form for this channel count (the
// contraction over channels in a kernel of its own, Gz[t] held in registers)
bool bwd_dst_split(int L, int C, bool bf16);
// channel count of its x layout: C padded to the kernel's ring turn
int bwd_dst_cpad(int C, bool bf16);
// Channels of the direct kernel's xd layout (d > 32): C rounded up to 64, 128
// or 256 (two, four or eight 32-channel tiles).
__host__ __device__ inline int bwd_direct_cpad(int C) { return C <= 64 ? 64 : (C <= 128 ? 128 : 256); }
hipError_t launch_bwd_dst(const BwdDstArgs& a, bool x_bf16, hipStream_t s);

// ---------------------------------------------------------------- misc
// Rank chunks (ranks above 256, split into column ranges):
// dst[row][j] = src[row][r0 + j] for a row-major [rows, R] src and [rows, n] dst
hipError_t launch_slice_cols(int rows, int R, int r0, int n, const float* src, float* dst, hipStream_t s);
// dst[row][r0 + j] = src[row][j]
hipError_t launch_scatter_cols(int rows, int R, int r0, int n, const float* src, float* dst, hipStream_t s);
// dst[i] += src[i], i < n
hipError_t launch_accumulate(size_t n, const float* src, float* dst, hipStream_t s);
// Compute units of the current device (cached per device).
int device_cus();
hipError_t launch_sh(int L, int E, const float* edge_vec, float* Y, float* dY, hipStream_t s);
hipError_t launch_zero(void* p, size_t bytes, hipStream_t s);

// ---------------------------------------------------------------- radial weights
// grad_Wrad[q, r] = sum_e phi_e[q] drho[e, r] (radial_grad.hip): per-block
// partial sums over fixed edge ranges, then their sum in block order.
int radial_grad_blocks(int E);
hipError_t launch_radial_grad(int E, int R, int n_radial, float sigma, const float* edge_vec, const float* drho,
                              float* partial, float* grad_radial_w, hipStream_t s);

// ---------------------------------------------------------------- radius graph
// Cell-list radius graph of a batch of systems (radius_graph.hip).
struct RadiusGraphArgs {
  int N, G;
  float r_cut;
  int max_neighbors;  // 0 = no cap
  int periodic[3];
  const float* pos;         // [N,3]
  const int32_t* graph_ptr; // [G+1]
  const float* cell;        // [G,3] (periodic axes only)
};
struct RadiusGraphLayout {
  size_t params, keys, gid, rank, flags, cell_off, spos, offs, tot, total;
  int n_keys;
};
RadiusGraphLayout radius_graph_layout(int N, int G);
// Maximum candidates (atoms and images within the cutoff) of one atom.
constexpr int kRadiusMaxNeighbours = 2048;
// Count pass: cells, atoms in cell order, per-atom neighbour counts, their
// prefix sum in ws.offs ([N+1], offs[N] = E) and the flags in ws.flags
// (int32: [0] graph_ptr invalid, [1] geometry invalid, [2] neighbour limit
// exceeded, [3] unused, [4] largest candidate count).
hipError_t launch_radius_count(const RadiusGraphArgs& a, char* ws, hipStream_t s);
// Emit pass (after the count pass on the same workspace; E = offs[N]).
hipError_t launch_radius_emit(const RadiusGraphArgs& a, char* ws, int max_candidates, int32_t* edge_index,
                              float* edge_vec, int32_t* edge_image, hipStream_t s);

}  // namespace tdn
