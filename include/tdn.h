/*
 * tdn.h -- C ABI of the MI355X (gfx950) CP tensor-product message-passing
 * layer of Tensor Decomposition Networks (arXiv 2507.01131).
 *
 * The layer replaces the Clebsch-Gordan tensor product of an equivariant
 * message-passing layer by its rank-R CP decomposition (Sec. 3.1, eq. cp and
 * eq. approximate) with one channel-mixing weight shared by every path
 * (Sec. 3.2).  For an edge e = (s, t) with vector r_e:
 *
 *   Y_e   = Y(r_e/|r_e|)              real spherical harmonics, degrees 0..L
 *   phi_e = exp(-(|r_e|-mu_q)^2/(2 sigma^2)),  mu_q = q r_cut/(n_radial-1),
 *           sigma = r_cut/(n_radial-1),  q = 0..n_radial-1
 *   g_e   = (B^T Y_e) * (phi_e radial_w)          (elementwise, length R)
 *   m_e   = D diag(g_e) A^T x[s] W                ([d, C])
 *   out[t] = sum over edges e into t of m_e
 *
 * Factor names: D is the output-mode factor (the paper's A), A acts on the
 * node features (the paper's B), B acts on the harmonics (the paper's C).
 *
 * Basis of the harmonics: index l*l + l + m (m = -l..l), real functions
 * without the Condon-Shortley phase, z the polar axis, m > 0 from
 * Re((x+iy)^m), m < 0 from Im((x+iy)^|m|), normalised so that Y_00 = 1 and
 * sum_m Y_lm^2 = 2l+1 on the unit sphere.
 *
 * Conventions for every entry point
 *  - Tensor pointers are DEVICE pointers owned by the caller, row-major and
 *    contiguous, 16-byte aligned.  The library allocates nothing; scratch
 *    space comes from the caller's workspace (size from tdn_workspace_size).
 *  - Work is enqueued asynchronously on `stream`; the return value reports
 *    argument validation and launch status.  With problem->validate = 1 the
 *    call also checks the edge data on the device and synchronises `stream`.
 *  - Outputs are overwritten, never accumulated.  A node without incoming
 *    edges gets a zero row.  E = 0 is valid.
 *  - Summation order is fixed (sorted-edge order, no floating-point
 *    atomics): repeated calls give bitwise identical results.
 *  - No exception or abort crosses the ABI.  Calls on different streams with
 *    different workspaces may run concurrently.
 */
#ifndef TDN_H
#define TDN_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TDN_OK = 0,
  TDN_ERR_NULL_POINTER = 1,        /* a required pointer is NULL                 */
  TDN_ERR_BAD_SHAPE = 2,           /* L, C, R, N, E, n_radial or r_cut invalid    */
  TDN_ERR_BAD_DTYPE = 3,           /* feat_dtype not a tdn_dtype                  */
  TDN_ERR_WORKSPACE_TOO_SMALL = 4, /* workspace_bytes below tdn_workspace_size    */
  TDN_ERR_INDEX_OUT_OF_RANGE = 5,  /* validate=1: src or dst outside [0, N)       */
  TDN_ERR_NOT_SORTED = 6,          /* validate=1: edges_sorted=1 but dst decreases */
  TDN_ERR_DEGENERATE_EDGE = 7,     /* validate=1: zero-length or non-finite r_e   */
  TDN_ERR_UNSUPPORTED_DEVICE = 8,  /* current device is not gfx950                */
  TDN_ERR_HIP = 9,                 /* a HIP call failed, see tdn_last_hip_error   */
  TDN_ERR_BAD_GEOMETRY = 10,       /* radius graph: graph_ptr, positions or box   */
  TDN_ERR_EDGE_CAPACITY = 11,      /* radius graph: more edges than buffer room   */
  TDN_ERR_NEIGHBOUR_LIMIT = 12,    /* radius graph: > 2048 candidates for an atom */
  TDN_ERR_SCRATCH_LIMIT = 13       /* no-allocation forward: workspace needed
                                      above TDN_NOALLOC_SCRATCH_BYTES           */
} tdn_status;

typedef enum { TDN_F32 = 0, TDN_BF16 = 1 } tdn_dtype;

typedef struct {
  int32_t L;            /* maximum degree, 0..6; d = (L+1)^2 components          */
  int32_t C;            /* channels (shared multiplicity), multiple of 16, <= 256  */
  int32_t R;            /* CP rank, 1..4096; ranks above 256 run as chunks of
                           consecutive rank columns whose per-node sums are added
                           in chunk order (the forward, backward and
                           no-allocation forward; the three-input product and
                           the atomics ablation take at most 256)            */
  int32_t n_nodes;      /* N >= 0                                                   */
  int32_t n_edges;      /* E >= 0 (E > 0 needs N > 0)                              */
  int32_t n_radial;     /* Gaussian radial functions, 2..16                        */
  float r_cut;          /* cutoff setting the Gaussian centres and width, > 0      */
  tdn_dtype feat_dtype; /* dtype of x and W (TDN_F32 or TDN_BF16); all else f32.
                           With TDN_BF16 the edge contractions run on bf16 MFMA:
                           the K operand g*A (and, in the backward, G W^T) is
                           rounded to bf16, accumulation stays fp32.  With
                           TDN_F32 results keep fp32-level accuracy (the
                           edge contractions run on 16-bit MFMA over exact
                           splits: two fp16 parts of power-of-two scaled
                           operands, or three bf16 parts)                    */
  int32_t edges_sorted; /* 1: edge_index already stably sorted by dst (perm is the
                           identity); 0: the call sorts                            */
  int32_t validate;     /* 1: check indices, order and edge vectors on the device */
} tdn_problem;

/* Workspace bytes needed by tdn_cp_tp_forward (*fwd_bytes) and
 * tdn_cp_tp_backward (*bwd_bytes); either pointer may be NULL.  The
 * workspace holds the intermediates of the CP layer of Sec. 3.1 and 3.2
 * (the per-node sums H_t and Z_t = D H_t, the operands in their MFMA
 * layouts, the destination sort) and of its backward, so its size follows
 * from N, E, L, C, R and n_radial alone.  The sizes
 * assume z_save == NULL (forward) and z_save == NULL (backward), i.e. the
 * largest case. */
tdn_status tdn_workspace_size(const tdn_problem* p, size_t* fwd_bytes, size_t* bwd_bytes);

/* Forward pass (Sec. 3.1 eq. approximate per edge, Sec. 3.2 shared W, summed
 * into the destination nodes).
 *   x          [N, d, C]  feat_dtype   node features, channel fastest
 *   edge_vec   [E, 3]     f32          r_e = pos[src] - pos[dst] (+ image shift)
 *   edge_index [2, E]     int32        row 0 = src, row 1 = dst
 *   A, B, D    [d, R]     f32          CP factors (constants)
 *   W          [C, C]     feat_dtype   out = Z W, W[c_in, c_out]
 *   radial_w   [n_radial, R] f32
 *   out        [N, d, C]  f32          overwritten
 *   z_save     [N, d, C]  f32 or NULL  Z = per-node sum of D diag(g) A^T x[s]
 *                                      (the layer before W), kept for backward
 *   perm       [E]        int32        sorted slot -> original edge id (stable
 *                                      by dst; ties keep the original order)
 *   offsets    [N+1]      int32        first sorted slot of each dst node,
 *                                      offsets[N] = E
 * perm and offsets are always written (bit-exact integer results). */
tdn_status tdn_cp_tp_forward(const tdn_problem* p, const void* x, const float* edge_vec,
                             const int32_t* edge_index, const float* A, const float* B,
                             const float* D, const void* W, const float* radial_w, float* out,
                             float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                             size_t workspace_bytes, hipStream_t stream);

/* Forward pass for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * Same arguments, results and bits as tdn_cp_tp_forward, without the
 * workspace: the scratch space comes from a fixed area of
 * TDN_NOALLOC_SCRATCH_BYTES that the library keeps on every device it runs
 * on until the process ends (set up on the first call on a device).  The
 * call allocates nothing.  A problem whose tdn_workspace_size forward bytes
 * exceed TDN_NOALLOC_SCRATCH_BYTES is rejected with TDN_ERR_SCRATCH_LIMIT
 * before any work is enqueued (molecules960_L3_C64_R64-sized problems fit;
 * the 3200-node headline size does not).  Every call on a device shares that
 * device's area, so calls that overlap on one device (other streams or host
 * threads) race: serialise them.  Records no timing events. */
#define TDN_NOALLOC_SCRATCH_BYTES (32u << 20)
tdn_status tdn_cp_tp_forward_noalloc(const tdn_problem* p, const void* x, const float* edge_vec,
                                     const int32_t* edge_index, const float* A, const float* B,
                                     const float* D, const void* W, const float* radial_w, float* out,
                                     float* z_save, int32_t* perm, int32_t* offsets, hipStream_t stream);

/* Measurement ablation of the forward's segmented sum (Sec. 3.1: the layer
 * sums the per-edge messages into each destination node).  Same arguments,
 * workspace and results as tdn_cp_tp_forward, within floating-point
 * reordering: the edge pass applies D to every edge's message on its own and
 * adds the d x C result into z_save (or the workspace's Z) with float atomics,
 * instead of summing each node's edges before one application of D and one
 * plain store.  The order of the additions is not fixed, so results may
 * differ between calls in the last bits.  Only fp32 features and 2 <= L <= 4
 * (TDN_ERR_BAD_DTYPE / TDN_ERR_BAD_SHAPE otherwise). */
tdn_status tdn_ablation_forward_atomics(const tdn_problem* p, const void* x, const float* edge_vec,
                                        const int32_t* edge_index, const float* A, const float* B,
                                        const float* D, const void* W, const float* radial_w,
                                        float* out, float* z_save, int32_t* perm, int32_t* offsets,
                                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The three-input CP product (App. A: an N-input multilinear map as
 * A (B1^T x1 * ... * BN^T xN), here N = 3 with the source node's features,
 * the edge's harmonics and the destination node's features):
 *   Z[t] = sum over edges e = (s, t) of D (g_e * (A^T x[s]) * (A2^T x[t])),
 *   g_e = (B^T Y_e) * (phi_e Wrad),   out = Z W.
 * Arguments as tdn_cp_tp_forward, plus A2 [d, R] f32, the factor of the
 * destination features; fp32 features and 2 <= L <= 4 only
 * (TDN_ERR_BAD_DTYPE / TDN_ERR_BAD_SHAPE); the same workspace size.  Since
 * A2^T x[t] is the same for every edge into t, it multiplies each node's
 * summed messages once. */
tdn_status tdn_cp_tp3_forward(const tdn_problem* p, const void* x, const float* edge_vec,
                              const int32_t* edge_index, const float* A, const float* A2, const float* B,
                              const float* D, const void* W, const float* radial_w, float* out, float* z_save,
                              int32_t* perm, int32_t* offsets, void* workspace, size_t workspace_bytes,
                              hipStream_t stream);

/* The attention block that consumes the CP messages (Sec. 4.1 "Model
 * Design": graph attention with MLP attention whose tensor products are the
 * CP product with path-weight sharing of Sec. 3.1 and 3.2).  The paper gives
 * no equations for the block; this is the reading implemented.  For an edge
 * e = (s, t):
 *   z_e  = D diag(g_e) A^T x[s]              the layer's message before W
 *   q_e  = [x[t]^(0), x[s]^(0), phi_e]       degree-0 rows and radial basis
 *   a_e  = LeakyReLU(q_e att_w1, 0.2) att_w2           [n_heads] logits
 *   alpha_e[h] = exp(a_e[h]) / sum over e' into t of exp(a_e'[h])
 *   out[t][:, c] = (sum over e into t of alpha_e[c / (C / n_heads)] z_e) W
 * Arguments as tdn_cp_tp_forward (fp32 features only, TDN_ERR_BAD_DTYPE),
 * and
 *   att_w1 [2C + n_radial, n_hidden] f32  rows: x[t]^(0) channels, x[s]^(0)
 *                                         channels, radial functions
 *   att_w2 [n_hidden, n_heads] f32
 *   alpha  [E, n_heads] f32 output: the weights by edge id (NULL: not stored)
 * 1 <= L <= 4, R <= 256, 1 <= n_heads <= 8 with C a multiple of
 * 32 n_heads, 1 <= n_hidden <= 64 (TDN_ERR_BAD_SHAPE otherwise).  The
 * weights' softmax runs over each destination's edges in sorted order with
 * its maximum subtracted; deterministic.  Workspace:
 * tdn_attention_workspace_size. */
tdn_status tdn_attention_workspace_size(const tdn_problem* p, int32_t n_heads, int32_t n_hidden, size_t* bytes);
tdn_status tdn_attention_forward(const tdn_problem* p, int32_t n_heads, int32_t n_hidden, const float* x,
                                 const float* edge_vec, const int32_t* edge_index, const float* A, const float* B,
                                 const float* D, const float* W, const float* radial_w, const float* att_w1,
                                 const float* att_w2, float* out, float* alpha, float* z_save, int32_t* perm,
                                 int32_t* offsets, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Measurement ablations of the forward's hot-path choices: the same layer
 * and arguments as tdn_cp_tp_forward (Sec. 3.1 eq. approximate, Sec. 3.2),
 * with one choice of the edge pass replaced (the paper attributes its speed
 * to this kind of kernel-level choice, Sec. 3.2 "coalesced memory access"):
 *   TDN_ABL_FACTORS_GLOBAL  the factor's packed operand blocks read in the
 *                           edge loop from a per-workgroup copy in global
 *                           memory instead of registers or LDS;
 *   TDN_ABL_Y_TABLE         the edge harmonics precomputed into a workspace
 *                           table by a kernel of their own and read by the
 *                           edge kernel instead of evaluated in it;
 *   TDN_ABL_VALU            the contraction, the segment sum and D in fp32
 *                           fused multiply-adds on the vector ALUs (one
 *                           workgroup per destination) instead of fp16 MFMA
 *                           over two-part splits; R <= 128, C <= 128.
 * fp32 features (TDN_ERR_BAD_DTYPE), 2 <= L <= 4 and R <= 256
 * (TDN_ERR_BAD_SHAPE, also for an unknown variant).  Results equal the
 * forward's to fp32 rounding (deterministic).  The workspace is
 * tdn_ablation_workspace_size's (the forward's plus the copies or the table).
 * Not for production use: they exist to be timed against the forward. */
#define TDN_ABL_FACTORS_GLOBAL 1
#define TDN_ABL_Y_TABLE 2
#define TDN_ABL_VALU 3
tdn_status tdn_ablation_workspace_size(const tdn_problem* p, int32_t variant, size_t* bytes);
tdn_status tdn_ablation_forward(const tdn_problem* p, int32_t variant, const void* x, const float* edge_vec,
                                const int32_t* edge_index, const float* A, const float* B, const float* D,
                                const void* W, const float* radial_w, float* out, float* z_save, int32_t* perm,
                                int32_t* offsets, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The exact CG tensor product over the same edges, as the comparator of the
 * CP layer (Sec. 2 eq. clebsch_gordan summed over every path (l1, l2, l3)
 * with l1, l2 <= L and |l1 - l2| <= l3 <= min(l1 + l2, L); Sec. 3.2 for the
 * per-path weight and the one channel weight W that all paths share):
 *   Z[n] = sum over edges e into n of K_e x[src_e],
 *   K_e[k, i] = sum_j C[k, i, j] Y_e[j] rho_e[path(k, i, j)],
 *   rho_e = phi_e path_w,   out = Z W.
 * Arguments as tdn_cp_tp_forward, with p->R the number of paths of degree L
 * (1, 5, 15, 34, 65, 111, 175 for L = 0..6; TDN_ERR_BAD_SHAPE otherwise) and
 * fp32 features only (TDN_ERR_BAD_DTYPE); the same workspace size.  The
 * coefficients C (device memory, read only) are rows over (k, i) pairs,
 * q = k d + i:
 *   cg_row [d*d + 1] int32   entries cg_row[q] .. cg_row[q+1] - 1 of row q
 *   cg_col [cg_nnz]  int32   j | path << 16 (path: index of the path in the
 *                            order l1, then l2, then l3 ascending)
 *   cg_val [cg_nnz]  f32     the coefficient
 *   path_w [n_radial, R] f32 radial weights of the paths
 * Rows are clamped to [0, cg_nnz] and entries with j >= d or path >= R are
 * skipped (a malformed table gives wrong values, never an out-of-bounds
 * read).  z_save, if not NULL, receives Z.  Deterministic: each node's edges
 * are summed in sorted order. */
tdn_status tdn_dense_tp_forward(const tdn_problem* p, const void* x, const float* edge_vec,
                                const int32_t* edge_index, const int32_t* cg_row, const int32_t* cg_col,
                                const float* cg_val, int32_t cg_nnz, const float* path_w, const void* W,
                                float* out, float* z_save, int32_t* perm, int32_t* offsets, void* workspace,
                                size_t workspace_bytes, hipStream_t stream);

/* The exact CG tensor product without path-weight sharing (the fully
 * connected product of Sec. 3.2: every path carries its own channel matrix,
 * applied to the path's block before the paths are summed):
 *   out[n]^(l3) = sum over edges e into n, paths p = (l1, l2, l3) of
 *                 rho_e[p] (C_p (x[src_e]^(l1) (x) Y_e^(l2))) W_paths[p],
 *   rho_e = phi_e path_w.
 * Since W_paths[p] acts on channels only, the kernel first sums each path's
 * block over a node's edges (N x (sum over paths of 2 l3 + 1) x C in the
 * workspace) and then applies the matrices per node.  Arguments as
 * tdn_dense_tp_forward, except:
 *   W_paths [R, C, C] f32   the channel matrix of each path, [in][out], paths
 *                           in the order l1, then l2, then l3 ascending
 * and no z_save.  fp32 features (TDN_ERR_BAD_DTYPE) and C <= 128
 * (TDN_ERR_BAD_SHAPE).  The path of an entry is its degree triple (deg i,
 * deg j, deg k); the table's path field is not read.  The workspace size is
 * tdn_dense_tp_unshared_workspace_size's.  Deterministic. */
tdn_status tdn_dense_tp_unshared_workspace_size(const tdn_problem* p, size_t* bytes);
tdn_status tdn_dense_tp_forward_unshared(const tdn_problem* p, const void* x, const float* edge_vec,
                                         const int32_t* edge_index, const int32_t* cg_row, const int32_t* cg_col,
                                         const float* cg_val, int32_t cg_nnz, const float* path_w,
                                         const float* W_paths, float* out, int32_t* perm, int32_t* offsets,
                                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Backward pass for the scalar <grad_out, out>.  perm and offsets are the
 * forward's outputs; z_save is the forward's saved Z or NULL (then Z is
 * recomputed).  Each gradient pointer may be NULL to skip it; grads are f32
 * for any feat_dtype:
 *   grad_x        [N, d, C]         dL/dx
 *   grad_W        [C, C]            dL/dW
 *   grad_edge_vec [E, 3]            dL/dr_e, in the caller's original edge order
 *   grad_radial_w [n_radial, R]     dL/dWrad = sum_e phi_e^T (dL/dg_e * v_e),
 *                                   summed in a fixed order (deterministic)
 * The CP factors are constants (no gradient; the paper caches them once per
 * L and keeps them fixed in training, Sec. 4.1). */
tdn_status tdn_cp_tp_backward(const tdn_problem* p, const void* x, const float* edge_vec,
                              const int32_t* edge_index, const float* A, const float* B,
                              const float* D, const void* W, const float* radial_w,
                              const int32_t* perm, const int32_t* offsets, const float* z_save,
                              const float* grad_out, float* grad_x, float* grad_W,
                              float* grad_edge_vec, float* grad_radial_w, void* workspace,
                              size_t workspace_bytes, hipStream_t stream);

/* Radius graph of a batch of atomic systems (App. "Model and Training
 * Configurations": the edges are built on the fly from a cutoff, with a cap
 * on the neighbours per atom -- 5.0 and 500 for OC20, 12.0 and 20 for OC22).
 * System g owns atoms graph_ptr[g] .. graph_ptr[g+1]-1; on a periodic axis a
 * it is a box of length cell[g][a] >= r_cut holding its atoms in [0, L).
 * Edge (src, dst, n), same system, source image n in {-1,0,1} per periodic
 * axis (0 elsewhere):
 *   r = (pos[src] - pos[dst]) + n * L      float32, each operation rounded
 *   kept when (rx*rx + ry*ry) + rz*rz < r_cut*r_cut (no fused multiply-add),
 *   except src == dst with n = 0,
 * so the edge set and vectors are exact functions of the float32 inputs.
 * max_neighbors > 0 keeps, per destination, the candidates smallest in
 * (|r|^2, src, image code).  Edges are ordered by (dst, src, image code),
 * code = (nx+1)*9 + (ny+1)*3 + (nz+1): edges_sorted = 1 input for
 * tdn_cp_tp_forward. */
typedef struct {
  int32_t n_nodes;       /* N atoms over all systems, 0 <= N < 2^26          */
  int32_t n_graphs;      /* G systems (>= 1 when N > 0)                      */
  float r_cut;           /* cutoff, > 0                                       */
  int32_t max_neighbors; /* 0 = no cap                                        */
  int32_t periodic[3];   /* 1 = the axis is periodic (every system)          */
} tdn_graph_problem;

tdn_status tdn_radius_graph_workspace_size(const tdn_graph_problem* g, size_t* bytes);

/*   pos        [N, 3]   f32    device
 *   graph_ptr  [G+1]    int32  device, graph_ptr[0] = 0, non-decreasing,
 *                              graph_ptr[G] = N
 *   cell       [G, 3]   f32    device box lengths (read on periodic axes
 *                              only; may be NULL when no axis is periodic)
 *   edge_index [2, E]   int32  row 0 = src, row 1 = dst (row stride E, the
 *                              edge count, not the capacity)
 *   edge_vec   [E, 3]   f32    r as above
 *   edge_image [E, 3]   int32  n (or NULL)
 *   offsets    [N+1]    int32  first edge of each dst, offsets[N] = E (or NULL)
 *   n_edges    host int64: E
 * edge buffers hold edge_capacity edges.  The call counts the edges first and
 * synchronises the stream once to read E and the checks; then, if
 * E <= edge_capacity, it writes the edges (asynchronously, on the stream).
 * E > edge_capacity returns TDN_ERR_EDGE_CAPACITY with *n_edges = E and
 * writes nothing (capacity 0 with NULL edge buffers asks for the count).
 * TDN_ERR_BAD_GEOMETRY: graph_ptr inconsistent, a non-finite position, a box
 * shorter than r_cut, or a periodic coordinate outside [0, L).
 * TDN_ERR_NEIGHBOUR_LIMIT: an atom has more than 2048 candidates within the
 * cutoff (before the cap).  Workspace from tdn_radius_graph_workspace_size;
 * not for capture in a HIP graph (it synchronises). */
tdn_status tdn_radius_graph(const tdn_graph_problem* g, const float* pos, const int32_t* graph_ptr,
                            const float* cell, int64_t edge_capacity, int32_t* edge_index,
                            float* edge_vec, int32_t* edge_image, int32_t* offsets, int64_t* n_edges,
                            void* workspace, size_t workspace_bytes, hipStream_t stream);

/* The grouping step of the layer's sum into destination nodes (the
 * out[t] sum above, taken over each destination's edges as one contiguous
 * segment so that the per-edge products of Sec. 3.1 eq. approximate are
 * summed in registers): a stable sort of the edges by destination,
 * exported for callers that sort once and pass edges_sorted = 1.
 * Stable sort of E integer keys in [0, n_keys): perm[p] = original index of
 * the p-th smallest key (equal keys keep their original order), offsets[k] =
 * number of keys < k, offsets[n_keys] = E.  Keys outside the range give
 * undefined perm/offsets (no memory fault).  Workspace from
 * tdn_sort_workspace_size. */
tdn_status tdn_sort_workspace_size(int32_t n_keys, int32_t E, size_t* bytes);
tdn_status tdn_sort_by_key(int32_t n_keys, int32_t E, const int32_t* keys, int32_t* perm,
                           int32_t* offsets, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/* The equivariant linear layer with path-weight sharing (Sec. 3.2, and its
 * use in the equivariant linear layers, Sec. 4.1 "Model Design"): one
 * channel matrix for every degree, y^(l) = x^(l) W for l = 0..L, i.e.
 *   y [N, d, C] = x [N, d, C] W [C, C]   (f32, channel fastest; W[c_in, c_out])
 * the map the layer applies to Z.  w_dtype TDN_F32 (fp32-level accuracy) or
 * TDN_BF16 (W in bf16 bits, x rounded to bf16 on the MFMA; fp32
 * accumulation).  Workspace from tdn_ps_linear_workspace_size (W's split
 * parts for TDN_F32, none for TDN_BF16).  n_nodes = 0 is a no-op; C in
 * 16..256 with C % 16 = 0, 0 <= L <= 6 (TDN_ERR_BAD_SHAPE). */
tdn_status tdn_ps_linear_workspace_size(int32_t C, int32_t w_dtype, size_t* bytes);
tdn_status tdn_ps_linear(int32_t n_nodes, int32_t L, int32_t C, const float* x, const void* W, int32_t w_dtype,
                         float* y, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Real spherical harmonics of edge directions (basis as above; the
 * harmonics input of the tensor product, Sec. 2, which the CP layer
 * contracts with its factor B, Sec. 3.1 eq. approximate), and their
 * Jacobian, which the backward uses for the gradient with respect to the
 * edge vectors:
 *   Y  [E, d]     Y(r_e/|r_e|)
 *   dY [E, d, 3]  dY/dr_e (or NULL) */
tdn_status tdn_spherical_harmonics(int32_t L, int32_t E, const float* edge_vec, float* Y,
                                   float* dY, hipStream_t stream);

/* Per-kernel timing with HIP events recorded on the launch stream.
 * tdn_timer_enable(1) starts recording every launch of the layer's edge
 * kernels; tdn_timer_read synchronises on the recorded events and returns
 * the summed milliseconds and launch count of the kernel named `kernel`
 * ("cp_edge_fwd", "cp_edge_fwd_att", "attention_weights", "cp_edge_fwd_atomic", "cp_edge_fwd_ablation",
 * "sh_table", "cp_edge_fwd_t3",
 * "dense_edge_fwd", "dense_edge_unshared",
 * "path_gemm", "radius_graph", "feature_layout",
 * "channel_layout", "cp_edge_bwd_src", "cp_bwd_dst", "radial_grad", "node_gemm", "gram",
 * "sort");
 * reset = 1 clears that kernel's record. */
tdn_status tdn_timer_enable(int32_t enable);
tdn_status tdn_timer_read(const char* kernel, double* total_ms, int32_t* launches, int32_t reset);

const char* tdn_status_string(tdn_status s);
int32_t tdn_last_hip_error(void); /* hipError_t behind the calling thread's last TDN_ERR_HIP */

#ifdef __cplusplus
}
#endif

#endif /* TDN_H */
