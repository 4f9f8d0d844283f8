/*
 * hg.h -- C ABI of libhg.so, the MI355X (gfx950) hot path of risk-aware
 * overlapping-subgraph GNN training.
 *
 * Paper: "Empowering Credit Risk Detection in Weixin Pay with Billion-Scale
 * Deep Graph Learning" (RAOS).  Each worker trains on one overlapping
 * subgraph; this library runs one worker's share on one GPU:
 *
 *   hg_build_csr            overlapping-subgraph construction (Methodology,
 *                           "Risk-Aware Subgraph Construction": candidate-set
 *                           and union equations; Algorithm 1, construction loop)
 *   hg_layer_fwd/_bwd       one relation-typed message-passing layer
 *                           (message, aggregation and update equations of the
 *                           "Heterogeneous Graph Transformer" paragraph, in the
 *                           relation-typed mean-aggregation form)
 *   hg_hgt_fwd/_bwd         the attention form of that layer: multi-head
 *                           mutual attention, per-destination softmax and
 *                           weighted aggregation (E6-E11)
 *   hg_mlp_bce_fwd_bwd,     the prediction head, masked BCE loss and Adam update
 *   hg_adam_step            of the joint objective (E18-E20)
 *   hg_temporal_fwd,        the temporal module: attention over the w previous
 *   hg_temporal_bwd         states and the GRU update (E12, E13)
 *   hg_align_loss_fwd_bwd   the CCA consistency-alignment loss on the overlap
 *                           nodes and its gradient (Section "Cross-Subgraph
 *                           Consistency Alignment", standardisation, invariance,
 *                           decorrelation and CCA-loss equations; the lambda_CCA
 *                           weight of the joint objective)
 *
 * Conventions (all entry points):
 *  - Pointers named in a struct or argument list are DEVICE pointers unless
 *    the comment says "host".  Matrices are row-major and contiguous.
 *  - The caller owns every buffer.  The library never allocates or frees
 *    device memory, keeps no pointer past a call and holds no mutable global
 *    state apart from a per-device property cache, the optional timing log
 *    (hg_timing_*) and the static device scratch of
 *    hg_align_loss_fwd_bwd_noalloc.  Calls on disjoint buffers are re-entrant.
 *  - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *    Everything except hg_build_csr is asynchronous on that stream.
 *  - Return value: HG_OK (0) or a negative HG_ERR_* code.  Arguments are
 *    validated on the host before any device work; on error nothing is
 *    launched (except HG_ERR_RANGE / HG_ERR_HIP, see hg_build_csr) and
 *    hg_last_error_detail() describes the cause.  No C++ exception crosses
 *    the ABI.
 *  - Ids are int32, counts int64, features float32 or bfloat16 (dtype),
 *    weights and weight gradients always float32.
 *  - Precision of the float32 dense products.  They run on the 16-bit MFMA
 *    with each float32 operand split into parts, a published way to recover
 *    float32 accuracy from 16-bit matrix units:
 *      row transforms (forward transforms, dX, the alignment's Grams and
 *      gradient, the temporal module's products with Q, Wi and Wh): the
 *      fp16 high part plus the fp16 remainder of each value,
 *      after scaling the row (and W) by a power of two so that its largest
 *      magnitude lies in [2^14, 2^15), with three of the four part
 *      products formed (Ootomo and Yokota, "Recovering single precision
 *      accuracy from Tensor Cores while surpassing the FP32 theoretical
 *      peak performance", IJHPCA 2022).  Each product term is exact to
 *      about 2^-21 of max|a row| x max|W| (the dropped remainder product
 *      and the rounded remainders), so a K-term dot product is within
 *      about K x 2^-21 x max|a| x max|w| of the exact value: float32
 *      rounding relative to the row's largest terms, not to each term, so
 *      a value much smaller than the largest of its row keeps fewer bits.
 *      weight gradients (split-K over rows): three bfloat16 parts per
 *      float32 value with the six part products of order at most two
 *      (Henry, Tang and Heinecke, "Leveraging the bfloat16 artificial
 *      intelligence datatype for higher-precision computations", ARITH
 *      2019): each product term relative to itself within about 2^-22;
 *      bfloat16 rows enter exactly.
 *    Sums are float32 (float64 where the kernel says so).
 */
#ifndef HG_H_
#define HG_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ------------------------------------------------------ */
#define HG_OK               0
#define HG_ERR_ARG         -1  /* null pointer, bad size or option          */
#define HG_ERR_RANGE       -2  /* an id >= n_nodes, rel >= n_rel, ntype >= n_ntype */
#define HG_ERR_CAPACITY    -3  /* workspace / plan too small (needed size in detail) */
#define HG_ERR_HIP         -4  /* a HIP runtime or launch error             */
#define HG_ERR_UNSUPPORTED -5  /* valid but not implemented (dtype, d, sizes) */

/* ---- options ----------------------------------------------------------- */
#define HG_KEY_OUTDEG  0   /* node key = out-degree over all relations      */
#define HG_KEY_HINDEX  1   /* node key = h-index of the out-neighbour multiset */
#define HG_KEYDIR_OUT  0   /* only direction implemented                    */
#define HG_THETA_NONE  2147483647
#define HG_DTYPE_F32   0
#define HG_DTYPE_BF16  1
#define HG_MAX_REL     255
#define HG_MAX_NTYPE   255

/* Input graph: one snapshot, typed nodes and typed directed edges
 * (Problem Formulation: node-type and edge-type maps).  Edge e goes from
 * src[e] to dst[e] with relation rel[e].  The base set is
 * V_k = { v : part[v] == k } (one block of the base partition, Graph
 * Partition paragraph).  Limits: 0 <= n_edges < 2^31, 1 <= n_nodes < 2^31,
 * n_nodes * n_rel < 2^31, 1 <= n_rel <= 255, 1 <= n_ntype <= 255. */
typedef struct hg_graph_desc {
  int64_t n_nodes;
  int64_t n_edges;
  int32_t n_rel;
  int32_t n_ntype;
  const int32_t* src;     /* [n_edges] */
  const int32_t* dst;     /* [n_edges] */
  const uint8_t* rel;     /* [n_edges] */
  const uint8_t* ntype;   /* [n_nodes] */
  const int32_t* part;    /* [n_nodes] partition id of every node */
  int32_t k;              /* this worker's partition */
  const float* edge_w;    /* [n_edges] message weight w_ij of each edge (the weighted
                           * edges of the problem formulation), or NULL = 1.  A
                           * message is multiplied by its weight; the mean's
                           * normaliser stays the in-edge count (reading A10). */
  /* Snapshots (end of "Risk-Aware Subgraph Construction": the snapshot
   * sequence is taken from the augmented subgraph by filtering on edge
   * timestamps).  With edge_ts != NULL the node set, the keys, the candidates
   * and the selection still use EVERY edge, and the induced subgraph keeps
   * only the edges with edge_ts[e] <= t_cut, so the snapshots of one
   * subgraph share local ids, overlap and type ranges.  NULL = no filter. */
  const int32_t* edge_ts; /* [n_edges] or NULL */
  int32_t t_cut;
  int32_t reserved;
} hg_graph_desc;

/* Budgeted long-tail overlap selection (h-index filter and TopM steps of
 * Algorithm 1).  Candidates C_k are nodes outside V_k joined to V_k by an
 * edge in either direction; C'_k keeps those with key <= theta; the first
 * min(budget_M, |C'_k|) of C'_k in ascending (key, splitmix64(seed ^ gid),
 * gid) order are selected, where splitmix64(x) is the first output of the
 * SplitMix64 generator (Steele, Lea and Flood 2014) started from state x. */
typedef struct hg_overlap_desc {
  int64_t budget_M;       /* >= 0 */
  int32_t key;            /* HG_KEY_OUTDEG or HG_KEY_HINDEX */
  int32_t key_dir;        /* HG_KEYDIR_OUT */
  int32_t theta;          /* >= 0; HG_THETA_NONE = no filter */
  int32_t reserved;
  uint64_t seed;
  /* NULL, or the key of every node [n_nodes] as hg_node_keys computes it
   * for this graph and key (device memory, read only).  Keys do not depend
   * on the partition block, so the builds of several blocks can share one
   * computation; the build then skips its own. */
  const int32_t* node_key;
} hg_overlap_desc;

/* Keys of every node of the graph (the selection key of the h-index filter
 * and TopM steps of Algorithm 1): keys[v] = out-degree of v over all
 * relations (HG_KEY_OUTDEG) or the h-index of the multiset of its
 * out-neighbours' out-degrees, one entry per edge (HG_KEY_HINDEX).  Uses
 * n_nodes, n_edges, n_rel, src, dst and rel of g; requires n_edges + n_nodes
 * < 2^31.  SYNCHRONOUS (like hg_build_csr); returns HG_ERR_RANGE when an
 * edge endpoint or relation is out of range (keys then unspecified).
 * keys int32 [n_nodes] is OVERWRITTEN.  ws: ws_bytes >=
 * hg_node_keys_workspace_size(g, key). */
size_t hg_node_keys_workspace_size(const hg_graph_desc* g, int32_t key);
int hg_node_keys(const hg_graph_desc* g, int32_t key, int32_t* keys, void* ws, size_t ws_bytes, void* stream);

/* Overlapping subgraph G[V_k u C_{k,M}] (union equation; induced subgraph of
 * Algorithm 1).  Local ids order the nodes by (node type, global id), so each
 * type is a contiguous range [type_off[t], type_off[t+1]).  Row (v, r) of the
 * CSR holds the in-edges of relation r of local node v (index v*n_rel + r),
 * entries in ascending original edge index; row (v, r) of the CSC holds the
 * out-edges of relation r of v, entries in ascending (destination, original
 * edge index).  csc_scale[p] = w / deg_r(csc_row[p]), the mean-aggregation
 * weight (w = the entry's edge weight, 1 without weights), as a correctly
 * rounded float32 quotient.
 *
 * The caller allocates every device array to CAPACITY: node arrays n_nodes,
 * overlap arrays min(budget_M, n_nodes), type_off n_ntype + 1, pointer arrays
 * n_nodes * n_rel + 1, edge arrays n_edges, plan hg_plan_size() bytes.
 * csr_eid may be NULL; csr_w may be NULL for a graph without weights.
 * hg_build_csr fills the host fields. */
typedef struct hg_subgraph {
  /* device outputs */
  int32_t* local2global;  /* [n_sub]  */
  int32_t* global2local;  /* [n_nodes], -1 for nodes outside the subgraph */
  int32_t* type_off;      /* [n_ntype + 1] */
  int32_t* overlap;       /* [m_sel] local ids of C_{k,M}, ascending */
  int32_t* overlap_home;  /* [m_sel] part[] of each overlap node */
  uint8_t* overlap_rel;   /* [m_sel] relation of the lowest-index edge joining it to V_k */
  int32_t* csr_ptr;       /* [n_sub * n_rel + 1] */
  int32_t* csr_col;       /* [e_sub] source local id */
  int32_t* csr_eid;       /* [e_sub] original edge index, or NULL */
  int32_t* csc_ptr;       /* [n_sub * n_rel + 1] */
  int32_t* csc_row;       /* [e_sub] destination local id */
  float*   csc_scale;     /* [e_sub] */
  float*   csr_w;         /* [e_sub] weight of each CSR entry; written for a weighted
                           * graph (required then), else unused and may be NULL */
  void*    plan;          /* opaque execution plan used by the layer kernels */
  size_t   plan_bytes;    /* capacity of plan */
  /* host outputs */
  int64_t n_nodes;        /* input graph sizes, copied from the descriptor */
  int64_t n_edges;
  int64_t n_sub;          /* |V_k u C_{k,M}| */
  int64_t e_sub;          /* edges of the induced subgraph */
  int64_t m_sel;          /* |C_{k,M}| */
  int32_t n_rel;
  int32_t n_ntype;
  int64_t type_off_host[HG_MAX_NTYPE + 1];
  int64_t n_active[HG_MAX_REL];   /* sources with >= 1 out-edge of relation r */
  int64_t plan_items;     /* backward work items (internal) */
  int64_t plan_heavy;     /* split CSC rows (internal) */
  int64_t plan_partials;  /* partial rows of split CSC rows (internal) */
  int64_t plan_fwd_heavy; /* destination rows split into chunks (internal) */
  int64_t plan_fwd_parts; /* chunks of those rows (internal) */
  int64_t plan_slot_rows; /* rows of the relation transforms in the layer workspaces (internal) */
  int64_t weighted;       /* 1 if built from a weighted graph (csr_w and csc_scale carry w) */
} hg_subgraph;

/* Bytes of `plan` for a graph with these input sizes. */
size_t hg_plan_size(int64_t n_nodes, int64_t n_edges, int32_t n_rel);

/* Scratch bytes hg_build_csr needs for this input (host call, no device work). */
size_t hg_build_csr_workspace_size(const hg_graph_desc* g, const hg_overlap_desc* o);

/* Build the overlapping subgraph of partition g->k.  SYNCHRONOUS: it
 * synchronises `stream` once at the end, checks the device-side range flag
 * and fills the host fields of *out.  Returns HG_ERR_RANGE if any src/dst is
 * outside [0, n_nodes), rel >= n_rel or ntype >= n_ntype (device arrays are
 * then unspecified).  ws: ws_bytes >= hg_build_csr_workspace_size(). */
int hg_build_csr(const hg_graph_desc* g, const hg_overlap_desc* o, hg_subgraph* out,
                 void* ws, size_t ws_bytes, void* stream);

/* One layer (the update equation with sigma = ReLU and the residual):
 *   z_j  = sum_r (1/|N_r(j)|) sum_{i in N_r(j)} h_i W_r + h_j W_self[type(j)] + b[type(j)]
 *   h'_j = (relu ? max(z_j, 0) : z_j) + (residual ? h_j : 0)
 * (an empty N_r(j) contributes 0).  d_in == d_out == d. */
typedef struct hg_layer_desc {
  int32_t d_in;
  int32_t d_out;
  int32_t dtype;     /* HG_DTYPE_F32 or HG_DTYPE_BF16 (feature storage); d in {64, 128, 256} */
  int32_t relu;      /* 0 or 1 */
  int32_t residual;  /* 0 or 1 */
} hg_layer_desc;

/* Bytes of `saved` (the ReLU mask: bit c of row j, at 32-bit word
 * j*(d/32) + c/32, bit c%32, is 1 iff z[j][c] > 0). */
size_t hg_layer_saved_size(const hg_subgraph* s, const hg_layer_desc* L);
size_t hg_layer_fwd_workspace_size(const hg_subgraph* s, const hg_layer_desc* L);
size_t hg_layer_bwd_workspace_size(const hg_subgraph* s, const hg_layer_desc* L);

/* Forward.  H_in, H_out: [n_sub, d] of dtype; W_rel [n_rel, d, d],
 * W_self [n_ntype, d, d] (row-vector convention y = x W), bias [n_ntype, d]
 * (may be NULL = 0).  saved receives the ReLU mask.  H_out must not alias H_in. */
int hg_layer_fwd(const hg_subgraph* s, const hg_layer_desc* L, const void* H_in,
                 const float* W_rel, const float* W_self, const float* bias,
                 void* H_out, void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward of hg_layer_fwd for upstream gradient dH_out = dL/dH_out:
 *   dZ = dH_out * mask,  dH_in = dH_out (residual) + dZ W_self^T + sum_r A_r^T dZ W_r^T,
 *   dW_r = (A_r H_in)^T dZ,  dW_self[t] = H_t^T dZ_t,  dbias[t] = sum_t dZ_t.
 * dH_in is OVERWRITTEN.  The weight gradients are OVERWRITTEN when
 * accumulate = 0 and added into when accumulate = 1 (weights shared by
 * several subgraphs: the sum over workers that the data-parallel gradient
 * all-reduce forms).  dbias may be NULL.  Deterministic: no floating-point
 * atomics, fixed reduction orders. */
int hg_layer_bwd(const hg_subgraph* s, const hg_layer_desc* L, const void* H_in,
                 const float* W_rel, const float* W_self, const void* saved,
                 const void* dH_out, void* dH_in, float* dW_rel, float* dW_self,
                 float* dbias, int32_t accumulate, void* ws, size_t ws_bytes, void* stream);

/* ---- heterogeneous graph transformer layer (E6-E11) ------------------------
 * S heads of width dk = d / S.  For an edge e = (i -> j) of relation r:
 *   K = H W_K[type] + b_K[type], Q = H W_Q[type] + b_Q[type], V = H W_V[type] + b_V[type]
 *   score^s(e) = (K^s_i W_att[r, s]) . Q^s_j * mu[type(i)][r][type(j)] / sqrt(dk)   (E6)
 *   msg^s(e)   = V^s_i W_msg[r, s]                                                   (E7)
 *   alpha^s(e) = softmax of score^s over the in-edges of j, all relations          (E8)
 *   h~_j       = concat_s sum_e alpha^s(e) msg^s(e)   (0 without in-edges)   (E9, E10)
 *   z_j = h~_j W_agg[type(j)] + b_agg[type(j)],
 *   h'_j = (relu ? max(z_j, 0) : z_j) + (residual ? h_j : 0)                       (E11)
 * x^s is columns [s dk, s dk + dk) of x.  Weights are float32 in the
 * row-vector convention: W_K, W_Q, W_V, W_agg [n_ntype, d, d]; b_K, b_Q, b_V,
 * b_agg [n_ntype, d] (each bias may be NULL = 0); W_att, W_msg
 * [n_rel, S, dk, dk]; mu [n_ntype, n_rel, n_ntype].  Passing W_V = W_K and
 * b_V = b_K makes the message reuse the key projection. */
typedef struct hg_hgt_desc {
  int32_t d;         /* 64 or 128 */
  int32_t heads;     /* S: d / S a power of two >= 4 */
  int32_t dtype;     /* HG_DTYPE_F32 */
  int32_t relu;      /* 0 or 1 */
  int32_t residual;  /* 0 or 1 */
  int32_t lean;      /* 0 or 1: `saved` leaves out the relation transforms of K
                        and V (about 5/7 of it at R = 5); the forward keeps them
                        in its workspace and the backward computes them again.
                        Sizes and results follow the flag; forward and backward
                        must be called with the same value. */
} hg_hgt_desc;

typedef struct hg_hgt_weights {
  const float *W_K, *b_K, *W_Q, *b_Q, *W_V, *b_V;
  const float *W_att, *W_msg, *mu;
  const float *W_agg, *b_agg;
} hg_hgt_weights;

/* Gradients, same shapes as hg_hgt_weights; all OVERWRITTEN.  A bias
 * gradient may be NULL (not computed). */
typedef struct hg_hgt_grads {
  float *W_K, *b_K, *W_Q, *b_Q, *W_V, *b_V;
  float *W_att, *W_msg, *mu;
  float *W_agg, *b_agg;
} hg_hgt_grads;

/* Bytes of `saved`: the forward's intermediates for the backward (K, Q, V,
 * the relation transforms of K and V, h~ and the per-head log-sum-exp of the
 * scores); its layout is internal.  The ReLU mask is a separate argument. */
size_t hg_hgt_saved_size(const hg_subgraph* s, const hg_hgt_desc* L);
size_t hg_hgt_fwd_workspace_size(const hg_subgraph* s, const hg_hgt_desc* L);
size_t hg_hgt_bwd_workspace_size(const hg_subgraph* s, const hg_hgt_desc* L);

/* Forward.  H_in, H_out: [n_sub, d] float32, H_out must not alias H_in.
 * mask [n_sub, d / 32] uint32 receives the ReLU decisions (bit c of row j at
 * word j*(d/32) + c/32, bit c%32, is 1 iff z[j][c] > 0; all ones when
 * relu = 0).  Asynchronous. */
int hg_hgt_fwd(const hg_subgraph* s, const hg_hgt_desc* L, const void* H_in, const hg_hgt_weights* W,
               void* H_out, void* mask, void* saved, void* ws, size_t ws_bytes, void* stream);

/* Backward of hg_hgt_fwd for dH_out = dL/dH_out, from the mask and `saved`
 * of the forward call with the same inputs (dZ = dH_out * mask).  dH_in
 * [n_sub, d] is OVERWRITTEN.  The weight gradients are OVERWRITTEN when
 * accumulate = 0 and added into when accumulate = 1 (a layer shared by the
 * snapshots of a sequence sums its per-snapshot gradients).  Deterministic:
 * no floating-point atomics. */
int hg_hgt_bwd(const hg_subgraph* s, const hg_hgt_desc* L, const void* H_in, const hg_hgt_weights* W,
               const void* mask, const void* saved, const void* dH_out, void* dH_in, const hg_hgt_grads* dW,
               int32_t accumulate, void* ws, size_t ws_bytes, void* stream);

/* CCA alignment on the overlap batch B (|B| = M):
 *   X = H[overlap] (local view), Y = H_ref (the other subgraph's view, row b
 *   for overlap[b]); per column mu and sigma = sqrt(var + eps), var with
 *   divisor M - ddof; Xh = (X - mu) / (sigma sqrt(M)), same for Y;
 *   L_inv = sum_b w_b ||Xh_b - Yh_b||^2 (w = 1 if NULL),
 *   L_dec = ||Xh^T Xh - I||_F^2 + ||Yh^T Yh - I||_F^2,  L = L_inv + lambda_n L_dec.
 * Writes loss3[0..2] = (L_inv, L_dec, L) (device float32) and writes
 * rows overlap[b] of dH as base[overlap[b]] + scale * dL/dX (scale =
 * lambda_CCA), base = dH_base when it is not NULL (then the other rows of
 * dH are untouched and dH_base is only read), else dH itself (the gradient
 * is ADDED into dH).  If dH_ref is not NULL it is OVERWRITTEN with
 * scale * dL/dY.  H, dH, dH_base: [n_rows, d]; H_ref, dH_ref: [M, d];
 * overlap entries distinct and in [0, n_rows).
 * M = 0 writes zeros.  Requires M > ddof, d in {64, 128, 256}.  dtype is
 * the storage type of H, H_ref, dH and dH_ref (float32 or bfloat16). */
size_t hg_align_workspace_size(int64_t M, int32_t d);
int hg_align_loss_fwd_bwd(int64_t M, int32_t d, int32_t dtype, int64_t n_rows,
                          const void* H, const int32_t* overlap, const void* H_ref,
                          const float* w, float lambda_n, float scale, float eps,
                          int32_t ddof, float* loss3, void* dH, const void* dH_base, void* dH_ref,
                          void* ws, size_t ws_bytes, void* stream);

/* The same alignment without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  The scratch lives in a static device
 * array of hg_align_noalloc_scratch_size() bytes (48 MiB) that every device
 * the library runs on holds until the process ends; it covers every batch
 * size at d <= 256 (the workspace of hg_align_loss_fwd_bwd is at most about
 * 43 MiB), and a call that would need more returns HG_ERR_CAPACITY.  The
 * call allocates nothing.  Arguments, results and errors are those of
 * hg_align_loss_fwd_bwd, bit for bit.  All calls on one device share its
 * scratch, which keeps the last call's contents (nothing in it has to start
 * at zero): calls that overlap on one device (other streams, other host
 * threads) race and must be serialised by the caller. */
size_t hg_align_noalloc_scratch_size(void);
int hg_align_loss_fwd_bwd_noalloc(int64_t M, int32_t d, int32_t dtype, int64_t n_rows,
                                  const void* H, const int32_t* overlap, const void* H_ref,
                                  const float* w, float lambda_n, float scale, float eps,
                                  int32_t ddof, float* loss3, void* dH, const void* dH_base, void* dH_ref,
                                  void* stream);

/* ---- prediction head, masked BCE and Adam ("Prediction and Optimization":
 * the two-layer MLP E18, the BCE loss E19, the joint objective E20) ---------
 *   a = H W1 + b1, hid = ReLU(a), o = hid W2 + b2, p = sigmoid(o)
 *   L_BCE = -(1/N_m) sum_{labels[i] >= 0} [y_i log p_i + (1 - y_i) log(1 - p_i)]
 * with y_i = labels[i] in {0, 1}; labels[i] = -1 marks an unlabelled row
 * (N_m = number of labelled rows; L_BCE = 0 and no gradient when N_m = 0).
 * H [n_rows, d], W1 [d, d_hidden], b1 [d_hidden], W2 [d_hidden, 1], b2 [1],
 * float32, row-vector convention; labels int8 [n_rows].  Writes loss[0]
 * (device), prob [n_rows] (p, may be NULL), OVERWRITES dH = dL_BCE/dH and
 * the weight gradients (db1, db2 may be NULL).  The joint objective adds
 * lambda_CCA * dL_CCA/dH with hg_align_loss_fwd_bwd into the same dH.
 * Requires d_hidden == d in {64, 128}; H, labels, dH may be NULL when
 * n_rows = 0.  Deterministic (fixed reduction order).
 * rows (may be NULL): int32 [n_list] distinct row indices in [0, n_rows)
 * that include every row with labels >= 0 (the labelled users, computed
 * once by the caller).  Only the listed rows go through the head -- the
 * loss and the gradients are those of the whole call, since an unlabelled
 * row contributes nothing -- and the other rows of dH are written as zero;
 * prob must then be NULL. */
size_t hg_mlp_bce_workspace_size(int64_t n_rows, int32_t d, int32_t d_hidden);
int hg_mlp_bce_fwd_bwd(int64_t n_rows, int32_t d, int32_t d_hidden, const float* H, const float* W1,
                       const float* b1, const float* W2, const float* b2, const int8_t* labels,
                       const int32_t* rows, int64_t n_list, float* loss, float* prob, float* dH, float* dW1,
                       float* db1, float* dW2, float* db2, void* ws, size_t ws_bytes, void* stream);

/* One Adam update (the optimiser paragraph; weight decay added to the
 * gradient, bias-corrected moments), in place on n float32 values:
 *   g = grad + weight_decay * param;  m = beta1 m + (1 - beta1) g;  v = beta2 v + (1 - beta2) g^2
 *   param -= lr * (m / (1 - beta1^step)) / (sqrt(v / (1 - beta2^step)) + eps)
 * step >= 1 counts updates (m = v = 0 before the first).  Asynchronous. */
int hg_adam_step(int64_t n, float* param, const float* grad, float* m, float* v, int64_t step, float lr,
                 float beta1, float beta2, float eps, float weight_decay, void* stream);

/* ---- temporal module ("Temporal Graph Learning": attention over the w
 * previous states E12, GRU update E13) ---------------------------------------
 * Per row (node) i, with c_0 .. c_{w-1} its w previous states, oldest first,
 * and h its spatial embedding at the current snapshot:
 *   u_k = tanh(Q c_k)  (Q applied to the column vector; row form c_k Q^T)
 *   s_k = r . u_k,  a = softmax_k(s),  Ht = sum_k a_k c_k                  (E12)
 *   g_r = sigmoid(h Wi[0] + bi[0] + Ht Wh[0] + bh[0])
 *   g_z = sigmoid(h Wi[1] + bi[1] + Ht Wh[1] + bh[1])
 *   g_n = tanh(h Wi[2] + bi[2] + g_r * (Ht Wh[2] + bh[2]))
 *   H   = (1 - g_z) * g_n + g_z * Ht                                        (E13)
 * w = 0 (no earlier state) gives Ht = 0.  Weights are float32: Q [d, d],
 * r [d], Wi, Wh [3, d, d] in the row-vector convention with the gates in the
 * order (reset, update, new) -- Wi[k] is the transpose of the k-th d x d
 * block of a GRU cell's stacked input weight, likewise Wh -- and bi, bh
 * [3, d] (either may be NULL = 0).  Rows (h, every c_k, H, dH, dh, dC_k) are
 * [n, d] in dtype (float32 or bfloat16).  C and dC are HOST arrays of w
 * DEVICE pointers.  Requires d = 64 and 0 <= w <= 4. */
typedef struct hg_temporal_weights {
  const float *Q, *r, *Wi, *bi, *Wh, *bh;
} hg_temporal_weights;

/* Gradients, same shapes as hg_temporal_weights.  bi and bh may be NULL
 * (not computed). */
typedef struct hg_temporal_grads {
  float *Q, *r, *Wi, *bi, *Wh, *bh;
} hg_temporal_grads;

/* Forward: writes H.  H must not alias h or a context state.  No workspace.
 * Asynchronous. */
int hg_temporal_fwd(int64_t n, int32_t d, int32_t w, int32_t dtype, const void* h, const void* const* C,
                    const hg_temporal_weights* W, void* H, void* stream);

/* Bytes of the backward workspace. */
size_t hg_temporal_bwd_workspace_size(int64_t n, int32_t d, int32_t w);

/* Backward of hg_temporal_fwd for dH = dL/dH (the forward is recomputed:
 * nothing is kept between the calls).  dh = dL/dh is OVERWRITTEN.  dL/dc_k is
 * ADDED into dC[k] (dC may be NULL, or any entry, for no gradient of that
 * state; callers zero a buffer before its first contribution), so one state
 * can collect the gradients of every later snapshot whose context holds it.
 * The weight gradients are OVERWRITTEN when accumulate = 0 and added into
 * when accumulate = 1 (weights shared over the snapshots).  dh and the dC[k]
 * must not alias each other or any input.  Deterministic: fixed reduction
 * orders, no floating-point atomics.  ws: ws_bytes >=
 * hg_temporal_bwd_workspace_size(n, d, w). */
int hg_temporal_bwd(int64_t n, int32_t d, int32_t w, int32_t dtype, const void* h, const void* const* C,
                    const hg_temporal_weights* W, const void* dH, void* dh, void* const* dC, int32_t accumulate,
                    const hg_temporal_grads* G, void* ws, size_t ws_bytes, void* stream);

/* ---- several subgraphs of one graph on one device (Algorithm 1 over K
 * workers) ---------------------------------------------------------------
 * The K overlapping subgraphs built by hg_build_csr from one graph with one
 * part[] (values in [0, K)) and k = 0 .. K-1 hold every node once as a base
 * node (in the subgraph of its own partition block) and once more in every
 * subgraph that selected it into its overlap.  These calls combine the
 * subgraphs' per-node rows.  g2l and h_parts are HOST arrays of K DEVICE
 * pointers: g2l[k] is subgraph k's global2local [n_nodes] (-1 = absent) and
 * h_parts[k] its rows [n_sub_k, d] in dtype (HG_DTYPE_F32 or HG_DTYPE_BF16,
 * float32 arithmetic); d in {64, 128, 256}; 1 <= K <= HG_MAX_PARTS.  All
 * three are asynchronous and deterministic (no atomics). */
#define HG_MAX_PARTS 64

/* MeanAgg (the inference step of Algorithm 1, and the averaging of an
 * overlap node's representations across workers in "Prediction and
 * Optimization"):
 *   H[v] = (1/cnt[v]) sum_{k : g2l[k][v] >= 0} h_parts[k][g2l[k][v]]
 * summed in k order, cnt[v] = number of those k.  A node in no subgraph gets
 * a zero row and cnt 0.  H [n_nodes, d] in dtype is OVERWRITTEN, as is cnt
 * int32 [n_nodes] (may be NULL).  H must not alias a subgraph's rows. */
int hg_mean_agg_fwd(int64_t n_nodes, int32_t d, int32_t dtype, int32_t K, const int32_t* const* g2l,
                    const void* const* h_parts, void* H, int32_t* cnt, void* stream);

/* Backward of hg_mean_agg_fwd into one subgraph with n_sub rows and
 * local2global l2g [n_sub]:  dh_part[i] = dH[l2g[i]] / cnt[l2g[i]],
 * OVERWRITTEN when accumulate = 0, added into when accumulate = 1.  cnt is
 * the forward's; a row whose node has cnt 0 (not possible for cnt from a
 * forward that included this subgraph) is written as NaN.  dH [n_nodes, d]
 * and dh_part [n_sub, d] in dtype; they must not alias. */
int hg_mean_agg_bwd(int64_t n_sub, int32_t d, int32_t dtype, const int32_t* l2g, const int32_t* cnt,
                    const void* dH, void* dh_part, int32_t accumulate, void* stream);

/* Home copies of one subgraph's overlap rows: the alignment target of an
 * overlap node is its representation in the subgraph of its own partition
 * block (Algorithm 1, the CCA term between a worker's overlap nodes and
 * their home copies):
 *   v = l2g[overlap[i]],  h = home[i],  Y[i] = h_parts[h][g2l[h][v]]
 * with overlap, home the subgraph's overlap [m] and overlap_home [m] and l2g
 * its local2global.  Y [m, d] in dtype is OVERWRITTEN; a row whose home is
 * outside [0, K) or whose node is absent from the home subgraph is written
 * as NaN.  On several devices this gather is the all-to-all exchange of the
 * overlap rows between the workers. */
int hg_home_gather(int64_t m, int32_t d, int32_t dtype, int32_t K, const int32_t* overlap, const int32_t* l2g,
                   const int32_t* home, const int32_t* const* g2l, const void* const* h_parts, void* Y,
                   void* stream);

/* ---- diagnostics ------------------------------------------------------- */
const char* hg_status_string(int status);
/* Thread-local description of the last error (host memory, valid until the
 * next call on this thread). */
const char* hg_last_error_detail(void);

/* ---- kernel timing (instrumentation, off by default) --------------------
 * While enabled, every kernel launch of this library is bracketed by two
 * hipEvents recorded on the launch stream.  hg_timing_collect synchronises
 * those events and returns, per kernel name, the number of launches and the
 * summed duration in milliseconds; it then clears the log. */
int hg_timing_enable(int on);
/* Fills up to `cap` entries; returns the number of kernel names (may exceed cap). */
int hg_timing_collect(char (*names)[64], int64_t* launches, double* total_ms, int cap);

#ifdef __cplusplus
}
#endif
#endif /* HG_H_ */
