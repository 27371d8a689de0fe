/*
 * pyg_mi355x.h -- C ABI of the MI355X (gfx950) message-passing library.
 *
 * The library computes the propagate path of PyTorch Geometric (Fey &
 * Lenssen, "Fast Graph Representation Learning with PyTorch Geometric",
 * 2019): an edge-parallel gather of source-node features followed by a
 * permutation-invariant scatter-reduce into target nodes, Eq. (1) of
 * Section 2 with gamma = identity, plus the preprocessing and readout steps
 * that use the same reduce.
 *
 * Graph format (Section 2, "Overview"): G = (X, (I, E)).
 *   x           node features [N, F], row-major, fp32 or bf16.
 *   edge_index  I in COO form, int64 [2, E], row-major: row 0 = source j,
 *               row 1 = target i; edge k carries phi(x_i, x_j, e_{j,i}) to i.
 *   edge_weight one scalar edge feature per edge (D = 1), fp32 [E], optional.
 *
 * Conventions shared by every call:
 *   - Every array pointer is a DEVICE pointer (hipMalloc'd, coarse-grained),
 *     owned by the caller. The library never allocates memory; scratch space
 *     comes from the caller through (ws, ws_bytes), sized by the matching
 *     *_workspace query. A too-small workspace returns PYG_ERR_WORKSPACE.
 *   - `stream` is a hipStream_t (NULL = the legacy default stream). All calls
 *     are asynchronous on that stream. Argument errors are detected on the
 *     host and returned before any device work is enqueued; PYG_ERR_HIP means
 *     a launch failed. Faults inside kernels surface at the caller's next
 *     synchronisation.
 *   - Outputs are fully overwritten, never accumulated into.
 *   - Node ids must lie in [0, N). Out-of-range ids are undefined behaviour
 *     unless rejected beforehand with pyg_validate_coo / pyg_validate_batch.
 *   - Sizes: N < 2^31 and E < 2^31 (int32 CSR columns and positions);
 *     larger sizes return PYG_ERR_UNSUPPORTED. N = 0, E = 0 or F = 0 are
 *     valid.
 *   - Calls are stateless and reentrant; concurrent calls on different
 *     streams must not share a workspace.
 */
#ifndef PYG_MI355X_H
#define PYG_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PYG_OK = 0,
    PYG_ERR_INVALID_ARG = -1, /* NULL / negative / inconsistent argument */
    PYG_ERR_INDEX_RANGE = -2, /* reserved for range failures reported by validation wrappers */
    PYG_ERR_WORKSPACE = -3,   /* ws_bytes below the *_workspace size */
    PYG_ERR_HIP = -4,         /* a HIP launch or runtime call failed */
    PYG_ERR_UNSUPPORTED = -5  /* size or combination outside the supported range */
} pyg_status;

typedef enum { PYG_F32 = 0, PYG_BF16 = 1 } pyg_dtype;

/* The permutation-invariant aggregation of Eq. (1): sum, mean or max. */
typedef enum { PYG_SUM = 0, PYG_MEAN = 1, PYG_MAX = 2 } pyg_aggr;

/* The message function phi of Eq. (1):
 *   PYG_MSG_SRC        phi = x_j, or w_k * x_j when a weight is given;
 *   PYG_MSG_DIFF       phi = x_j - x_i (the EdgeConv message, Section 2);
 * and, with F-dimensional edge features e_{j,i} (pyg_propagate_edge only):
 *   PYG_MSG_EDGE_ADD   phi = x_j + e_{j,i};
 *   PYG_MSG_EDGE_RELU  phi = max(x_j + e_{j,i}, 0) (GINE-style);
 *   PYG_MSG_EDGE_MUL   phi = x_j * e_{j,i}, elementwise. */
typedef enum {
    PYG_MSG_SRC = 0,
    PYG_MSG_DIFF = 1,
    PYG_MSG_EDGE_ADD = 2,
    PYG_MSG_EDGE_RELU = 3,
    PYG_MSG_EDGE_MUL = 4
} pyg_msg;

/* Kernel choice (Appendix A contrasts the two schemes):
 *   PYG_KERNEL_COO_ATOMIC   gather/scatter over the unsorted COO with
 *                           hardware atomics; needs no preprocessing;
 *   PYG_KERNEL_CSR_SEGMENT  target-sorted (CSR) segment reduction; needs the
 *                           CSR built once by pyg_coo_to_csr; deterministic;
 *   PYG_KERNEL_AUTO         CSR when a CSR is passed, else COO. */
typedef enum { PYG_KERNEL_AUTO = 0, PYG_KERNEL_COO_ATOMIC = 1, PYG_KERNEL_CSR_SEGMENT = 2 } pyg_kernel;

/* Order of per-edge arrays [E, H] of the attention calls:
 *   PYG_ORDER_CSR  indexed by CSR slot (coalesced; what pyg_propagate_heads reads);
 *   PYG_ORDER_COO  indexed by COO edge id, reached through csr->perm. */
typedef enum { PYG_ORDER_CSR = 0, PYG_ORDER_COO = 1 } pyg_order;

/* A target-sorted CSR built by pyg_coo_to_csr (device pointers).
 *   rowptr [N+1]  rowptr[i]..rowptr[i+1] are the CSR slots of target i;
 *   col    [E]    source node of each slot;
 *   perm   [E]    COO edge id of each slot (ascending inside a row);
 *   weight [E]    CSR-ordered edge weight, or NULL when unweighted;
 *   chunk         edges per work unit of the segment kernel, 0 = default. */
typedef struct {
    const int64_t *rowptr;
    const int32_t *col;
    const int64_t *perm;
    const float *weight;
    int64_t N;
    int64_t E;
    int64_t chunk;
} pyg_csr;

/* A CSR whose slots are regrouped by source block (built by
 * pyg_csr_blocks_build from a pyg_csr): the source ids are cut into B blocks
 * of ceil(N / B) consecutive ids, and virtual row b * N + i holds the slots
 * of target i whose source lies in block b, in ascending edge id. It is a
 * CSR over B * N rows:
 *   rowptr [B*N + 1]  rowptr[b*N + i] .. rowptr[b*N + i + 1];
 *   col    [E]        source node of each slot;
 *   perm   [E]        COO edge id of each slot, or NULL (needed for max);
 *   weight [E]        edge weight in this slot order, or NULL;
 *   B                 2 .. 32;
 *   chunk             slots per work unit of the propagate, 0 = default. */
typedef struct {
    const int64_t *rowptr;
    const int32_t *col;
    const int64_t *perm;
    const float *weight;
    int64_t N;
    int64_t E;
    int64_t B;
    int64_t chunk;
} pyg_csr_blocks;

/* Human-readable text for a status code (static storage, never NULL). */
const char *pyg_strerror(int status);

/* ABI version of this header (incremented on incompatible change). */
int pyg_abi_version(void);

/* Workspace bytes needed by pyg_degree for (E, N). */
int pyg_degree_workspace(int64_t E, int64_t N, size_t *bytes);

/* In-degree deg[i] = number of edges whose target is i, counted with
 * multiplicity (|N(i)| in Eq. (1); the denominator of mean).
 *   edge_index int64 [2,E] (device), deg int64 [N] (device, output).
 * Counted in on-chip histograms over slices of the node range; exact.
 * Errors: PYG_ERR_INVALID_ARG (negative sizes, NULL arrays, E > 0 with
 * N = 0), PYG_ERR_UNSUPPORTED (N or E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_degree(const int64_t *edge_index, int64_t E, int64_t N, int64_t *deg, void *ws, size_t ws_bytes,
               void *stream);

/* In-degree (|N(i)| in Eq. (1)) from a CSR built by pyg_coo_to_csr:
 * deg[i] = rowptr[i+1] - rowptr[i], the same counts as pyg_degree on the
 * edge list the CSR was built from (its rows are the targets), read off the
 * row boundaries the sort produced instead of counting the edge list again.
 *   csr  read: rowptr and N only;  deg  int64 [N] (device, output).
 * Errors: PYG_ERR_INVALID_ARG (NULL csr or rowptr, N < 0, NULL deg with
 * N > 0). */
int pyg_degree_csr(const pyg_csr *csr, int64_t *deg, void *stream);

/* Workspace bytes needed by pyg_coo_to_csr for (E, N). */
int pyg_coo_to_csr_workspace(int64_t E, int64_t N, size_t *bytes);

/* Target-sorted CSR of the COO edge list (the row-ordered, "coalesced"
 * layout of Appendix A, built once as preprocessing). The sort is stable:
 * inside a row the slots keep ascending COO edge id, so the result is
 * unique and bit-reproducible.
 *   edge_index  int64 [2,E]        input;
 *   edge_weight fp32 [E] or NULL   input, COO order;
 *   rowptr      int64 [N+1]        output;
 *   col         int32 [E]          output;
 *   perm        int64 [E]          output;
 *   weight_csr  fp32 [E] or NULL   output, = edge_weight[perm] (requires
 *                                  edge_weight, ignored when it is NULL).
 * Errors: PYG_ERR_INVALID_ARG (negative sizes, NULL rowptr, or NULL
 * edge_index/col/perm or N = 0 when E > 0), PYG_ERR_UNSUPPORTED (N or
 * E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_coo_to_csr(const int64_t *edge_index, int64_t E, int64_t N, const float *edge_weight,
                   int64_t *rowptr, int32_t *col, int64_t *perm, float *weight_csr,
                   void *ws, size_t ws_bytes, void *stream);

/* CSR-ordered copy of a COO-ordered edge array: out[p] = in[perm[p]] for
 * p < E, with perm from pyg_coo_to_csr (e.g. fresh edge weights for an
 * existing CSR). in and out are fp32 [E] device arrays and must differ.
 * Errors: PYG_ERR_INVALID_ARG (E < 0, NULL arrays, in == out),
 * PYG_ERR_UNSUPPORTED (E >= 2^31). */
int pyg_gather_edges(const int64_t *perm, int64_t E, const float *in, float *out, void *stream);

/* Workspace bytes needed by pyg_gcn_norm for (E, N). */
int pyg_gcn_norm_workspace(int64_t E, int64_t N, size_t *bytes);

/* GCN edge normalisation for the GCN operator of Section 2, on an edge list
 * that already contains the self-loops:
 *   d_i = sum of w_k over edges with target i (w = 1 when edge_weight is NULL),
 *   norm_k = d_j^-1/2 * w_k * d_i^-1/2 for edge k = (j -> i), 0 where d = 0.
 * Computed in fp64 and rounded once to fp32.
 *   deg  int64 [N] or NULL: the in-degree of this edge list as returned by
 *        pyg_degree, reused instead of counting again; read only when
 *        edge_weight is NULL (weighted degrees are always summed here);
 *   norm fp32 [E] output in COO order.
 * Errors: PYG_ERR_INVALID_ARG (negative sizes, NULL edge_index/norm or
 * N = 0 when E > 0), PYG_ERR_UNSUPPORTED (N or E >= 2^31),
 * PYG_ERR_WORKSPACE. */
int pyg_gcn_norm(const int64_t *edge_index, const float *edge_weight, int64_t E, int64_t N,
                 const int64_t *deg, float *norm, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_gcn_norm_csr for N nodes. */
int pyg_gcn_norm_csr_workspace(int64_t N, size_t *bytes);

/* The same GCN normalisation computed on a CSR from pyg_coo_to_csr and
 * written in CSR slot order, ready to serve as csr->weight of a propagate:
 *   d_i = sum of the weights of row i's slots (csr->weight, or 1 when NULL),
 *   norm_csr[p] = d_j^-1/2 * w_p * d_i^-1/2 for slot p of row i, j = col[p].
 * Equal to pyg_gcn_norm's output gathered through csr->perm: bit for bit
 * with unit weights; with weights the fp64 degree sums are ordered per row
 * (deterministic) and may differ from another order by one fp32 ulp.
 *   norm_csr fp32 [E] output (device).
 * Errors: PYG_ERR_INVALID_ARG (NULL csr/rowptr, negative sizes, NULL
 * col/norm_csr or N = 0 when E > 0), PYG_ERR_UNSUPPORTED (N or E >= 2^31),
 * PYG_ERR_WORKSPACE. */
int pyg_gcn_norm_csr(const pyg_csr *csr, float *norm_csr, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_gcn_propagate (chunk = csr->chunk). */
int pyg_gcn_propagate_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t chunk, size_t *bytes);

/* The GCN propagate with its normalisation fused in (the GCN operator of
 * Section 2; Eq. (1) with phi = norm_p * x_j and a sum):
 *   out[i] = sum over the slots p of row i of norm_p * x[col[p]],
 *   norm_p = d_j^-1/2 * w_p * d_i^-1/2, d and w as pyg_gcn_norm_csr (the CSR's
 * weights, or 1), formed in fp64 and rounded once to fp32 per slot inside
 * the propagate (by its first 128-byte feature window, which writes them;
 * the later windows read them back), instead of a separate pass.
 *   csr       CSR from pyg_coo_to_csr; csr->weight optional (the w_p);
 *   norm_out  fp32 [E] in CSR slot order, or NULL: receives every norm_p,
 *             equal bit for bit to pyg_gcn_norm_csr's output;
 *   x, out    as pyg_propagate (out fully overwritten, fp32 accumulation).
 * Deterministic. Errors: PYG_ERR_INVALID_ARG (bad dtype, NULL/inconsistent
 * csr, NULL x/out, norm_out or out overlapping another array),
 * PYG_ERR_UNSUPPORTED (N or E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_gcn_propagate(const void *x, int dtype, int64_t N, int64_t F, const pyg_csr *csr, float *norm_out,
                      void *out, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_propagate for this shape, aggregation and
 * kernel (pass the same chunk as csr->chunk; 0 = default). */
int pyg_propagate_workspace(int dtype, int64_t N, int64_t F, int64_t E, int aggr, int kernel,
                            int64_t chunk, size_t *bytes);

/* Propagate, Eq. (1) of Section 2 with gamma = identity:
 *   out[i, f] = AGG over edges k = (j -> i) of phi_k[f],
 * phi from `msg` (w_k * x_j when a weight is given), AGG from `aggr`.
 *   x           [N,F] fp32 or bf16 (dtype), 16-byte aligned rows give the
 *               vector path (F * sizeof(dtype) % 16 == 0), otherwise scalar;
 *   edge_index  [2,E] COO (required by the COO kernel; may be NULL for CSR);
 *   edge_weight fp32 [E] COO order or NULL, read by the COO kernel. The CSR
 *               kernel reads the weights from csr->weight instead (the call
 *               is weighted when csr->weight is set; edge_weight without
 *               csr->weight is an error). Weights are not allowed with
 *               PYG_MSG_DIFF;
 *   csr         CSR from pyg_coo_to_csr or NULL;
 *   out         [N,F] in x's dtype; fp32 accumulation, one rounding to bf16;
 *   argmax      int64 [N,F], required for PYG_MAX and NULL otherwise: the COO
 *               edge id of the winning message.
 * Semantics: an empty neighbourhood gives 0 and argmax = E. mean divides by
 * the number of incoming edges. max compares fp32 messages with -0.0 taken
 * as +0.0; equal maxima resolve to the lowest edge id. Max, argmax and every
 * CSR result are bit-reproducible; COO sum/mean use float atomics and may
 * differ in the last bits between runs (Appendix A notes the same of GPU
 * scatter). `out` must not overlap `x`.
 * Errors: PYG_ERR_INVALID_ARG (bad dtype/msg/aggr/kernel, negative
 * sizes, NULL arrays, argmax given without max or missing with it, a weight
 * with difference messages, out overlapping x, a CSR that does not match
 * N, E or the weights, CSR_SEGMENT without a CSR), PYG_ERR_UNSUPPORTED (N or
 * E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_propagate(const void *x, int dtype, int64_t N, int64_t F,
                  const int64_t *edge_index, int64_t E, const float *edge_weight,
                  const pyg_csr *csr, int msg, int aggr, int kernel,
                  void *out, int64_t *argmax, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_csr_blocks_build. */
int pyg_csr_blocks_workspace(int64_t N, int64_t E, int64_t B, size_t *bytes);

/* Regroups the slots of a CSR (pyg_coo_to_csr) by source block, for
 * pyg_propagate_blocked: the preprocessing of the same row-ordered layout
 * Appendix A builds once per graph, cut by source as well so that the
 * propagate's wavefronts in flight gather from one source block (a 1/B part
 * of x) at a time. Stable: inside a virtual row the
 * slots keep the CSR's order (ascending edge id), so the result is unique.
 *   csr     input CSR (rowptr, col; perm when perm is wanted, weight when
 *           weight is wanted);
 *   B       source blocks, 2 .. 32;
 *   rowptr  int64 [B*N + 1] output;  col  int32 [E] output;
 *   perm    int64 [E] output or NULL (COO edge id of every slot);
 *   weight  fp32 [E] output or NULL (csr->weight in the new slot order).
 * Errors: PYG_ERR_INVALID_ARG (NULL csr/rowptr/col, a bad B, perm or weight
 * wanted but absent from csr), PYG_ERR_UNSUPPORTED (N or E >= 2^31),
 * PYG_ERR_WORKSPACE. */
int pyg_csr_blocks_build(const pyg_csr *csr, int64_t B, int64_t *rowptr, int32_t *col, int64_t *perm,
                         float *weight, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_coo_to_csr_blocked. */
int pyg_coo_to_csr_blocked_workspace(int64_t E, int64_t N, int64_t B, size_t *bytes);

/* The source-blocked CSR straight from the COO (the same arrays as
 * pyg_csr_blocks_build(pyg_coo_to_csr(...)), bit for bit, in one sort):
 * the stable radix sort of pyg_coo_to_csr keyed by the virtual row
 * (source / ceil(N / B)) * N + target instead of the target, so that slots
 * are ordered by source block, then target, then edge id. The
 * preprocessing of Appendix A's row-ordered layout in the form that the
 * blocked propagate reads; with B * N below 2^31.
 *   edge_index, E, N, edge_weight  as pyg_coo_to_csr;
 *   B       source blocks, 2 .. 32;
 *   rowptr  int64 [B*N + 1] output; col int32 [E] output;
 *   perm    int64 [E] output or NULL (the COO edge id of every slot; needed
 *           by max);
 *   weight_csr fp32 [E] output or NULL (edge_weight in the blocked order).
 * Errors: PYG_ERR_INVALID_ARG (negative sizes, a bad B, NULL rowptr, NULL
 * edge_index/col or N = 0 when E > 0), PYG_ERR_UNSUPPORTED (N, E or B*N >=
 * 2^31), PYG_ERR_WORKSPACE. */
int pyg_coo_to_csr_blocked(const int64_t *edge_index, int64_t E, int64_t N, int64_t B, const float *edge_weight,
                           int64_t *rowptr, int32_t *col, int64_t *perm, float *weight_csr, void *ws,
                           size_t ws_bytes, void *stream);

/* In-degree from a source-blocked CSR: deg[i] = the slots of target i over
 * all blocks (bit-exact; equal to pyg_degree).
 *   deg int64 [N] output. Errors: PYG_ERR_INVALID_ARG (NULL bcsr/rowptr/deg,
 * a bad B). */
int pyg_degree_csr_blocks(const pyg_csr_blocks *bcsr, int64_t *deg, void *stream);

/* Workspace bytes needed by pyg_propagate_blocked (chunk as in the blocked
 * CSR). Holds B fp32 partial rows per target (B*N*F*4 bytes, plus B*N*F*8
 * for max). */
int pyg_propagate_blocked_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t B, int aggr, int64_t chunk,
                                    size_t *bytes);

/* Propagate (Eq. (1) of Section 2, the same results as pyg_propagate with
 * the CSR kernel) over a source-blocked CSR: the virtual rows are reduced
 * into fp32 partial rows one 128-byte feature window at a time, block after
 * block inside a window (so the rows of x gathered at any moment are one
 * window of one source block, which the L2s hold far better than a window
 * of all of x), and the partials of each target are then folded in block
 * order. Sum and mean differ from pyg_propagate only in the
 * order of the additions (deterministic, the same tolerance); max and argmax
 * are the same bits (ties to the lowest edge id across blocks too).
 *   x    [N,F] fp32 or bf16 with 16-byte rows (F * sizeof(dtype) % 16 == 0)
 *        and 16-byte aligned x and out;
 *   bcsr from pyg_csr_blocks_build (weighted when bcsr->weight is set; perm
 *        required for max);
 *   msg  PYG_MSG_SRC or PYG_MSG_DIFF (no weight with DIFF); aggr, out,
 *        argmax as pyg_propagate.
 * Errors: as pyg_propagate, plus PYG_ERR_UNSUPPORTED for rows that are not
 * 16-byte vectors or a bad B. */
int pyg_propagate_blocked(const void *x, int dtype, int64_t N, int64_t F, const pyg_csr_blocks *bcsr, int msg,
                          int aggr, void *out, int64_t *argmax, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_gcn_propagate_blocked (chunk as in the
 * blocked CSR): d^-1/2, the norms when norm_out is NULL, fp32 rows of
 * d^-1/2 x (fp32 only), and the blocked propagate's partial rows. */
int pyg_gcn_propagate_blocked_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t B, int64_t chunk,
                                        size_t *bytes);

/* pyg_gcn_propagate over a source-blocked CSR (the GCN operator of Section
 * 2 with the normalisation fused in, on the blocked schedule of
 * pyg_propagate_blocked):
 *   out[i] = sum over the edges (j -> i) of norm * x[j],
 *   norm = d_j^-1/2 * w * d_i^-1/2, d from `csr` exactly as
 * pyg_gcn_norm_csr takes it (row lengths, or csr->weight summed in fp64 in
 * CSR slot order) when csr is given, else from bcsr (the row lengths summed
 * over the blocks, or the weights summed in fp64 in blocked slot order),
 * formed in fp64 and rounded once per slot. When norm_out is given, the
 * first 128-byte feature window forms these norms, uses them and writes
 * them. For fp32 rows the other windows (all of them when norm_out is NULL)
 * instead sum w * (d_j^-1/2 x_j) (the rows pre-scaled in the workspace, an
 * fp64 product rounded once) and the fold multiplies by d_i^-1/2 in fp64:
 * the same sum up to rounding, with no per-slot norm; for bf16 rows they
 * read the norms back.
 *   csr       the graph's CSR (pyg_coo_to_csr), for d, or NULL;
 *   bcsr      pyg_csr_blocks_build(csr, ...) or pyg_coo_to_csr_blocked,
 *             weighted iff csr is weighted;
 *   norm_out  fp32 [E] in bcsr's slot order, or NULL: every norm, equal bit
 *             for bit to pyg_gcn_norm_csr's norm of the same edge (with
 *             weights and csr NULL: up to the order of the fp64 degree sum);
 *   x, out    as pyg_propagate_blocked (16-byte rows; out overwritten).
 * Sum differs from pyg_gcn_propagate only in the order of the additions
 * (deterministic). Errors: PYG_ERR_INVALID_ARG (bad dtype, NULL bcsr,
 * mismatched csr/bcsr, NULL x/out, overlapping arrays), PYG_ERR_UNSUPPORTED
 * (N or E >= 2^31, rows that are not 16-byte vectors), PYG_ERR_WORKSPACE. */
int pyg_gcn_propagate_blocked(const void *x, int dtype, int64_t N, int64_t F, const pyg_csr *csr,
                              const pyg_csr_blocks *bcsr, float *norm_out, void *out, void *ws, size_t ws_bytes,
                              void *stream);

/* Size of the static scratch array of pyg_propagate_noalloc, per GPU. */
#define PYG_NOALLOC_SCRATCH_MIB 128

/* pyg_propagate without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc). Same arguments, kernels, results
 * and errors as pyg_propagate, minus (ws, ws_bytes): the scratch comes from
 * a static device array of PYG_NOALLOC_SCRATCH_MIB MiB that every GPU the
 * library runs on holds until the process ends. The call allocates nothing.
 *   stream  must belong to the current device (else PYG_ERR_INVALID_ARG);
 *           the current device's array is used.
 * A call that needs more scratch than the array holds (pyg_propagate_workspace
 * above PYG_NOALLOC_SCRATCH_MIB MiB, e.g. max on graphs of ~10^8 edges)
 * returns PYG_ERR_UNSUPPORTED before any device work. Every call on one GPU
 * shares that GPU's array: calls that overlap in time on one GPU (two
 * streams, two host threads) race and give wrong results; calls ordered on
 * one stream are safe, whatever an earlier call left in the array.
 * PYG_ERR_HIP if the device or the array's address cannot be queried. */
int pyg_propagate_noalloc(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                          const float *edge_weight, const pyg_csr *csr, int msg, int aggr, int kernel, void *out,
                          int64_t *argmax, void *stream);

/* Propagate with F-dimensional edge features in the message (Eq. (1)'s
 * e_{j,i}; Section 2 and Appendix A name the integration of
 * multi-dimensional edge information as a property of the gather/scatter
 * scheme):
 *   out[i, f] = AGG over edges k = (j -> i) of phi(x_j[f], e_k[f]),
 * phi from msg (PYG_MSG_EDGE_ADD / _RELU / _MUL), AGG from aggr.
 *   edge_attr  [E, F] in x's dtype (device); attr_order PYG_ORDER_COO (row k
 *              = edge k) or PYG_ORDER_CSR (row p = CSR slot p, the coalesced
 *              layout; CSR kernel only, COO order is reached through
 *              csr->perm);
 *   kernel     as in pyg_propagate (COO atomics or CSR segments); the CSR
 *              kernel ignores csr->weight here;
 *   other arguments, the workspace (pyg_propagate_workspace), outputs,
 *   argmax, tie and -0.0 rules as in pyg_propagate. Messages are formed in
 *   fp32 (one add or multiply, then max(., 0) for _RELU); max compares them.
 * Errors: as pyg_propagate, plus PYG_ERR_INVALID_ARG for a message other
 * than the three edge messages, a bad attr_order, or NULL edge_attr. */
int pyg_propagate_edge(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                       const void *edge_attr, int attr_order, const pyg_csr *csr, int msg, int aggr, int kernel,
                       void *out, int64_t *argmax, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_propagate_edge_encoded (kernel as passed to
 * the call; chunk = csr->chunk for the CSR kernel, else 0). */
int pyg_propagate_edge_encoded_workspace(int dtype, int64_t N, int64_t F, int64_t E, int64_t D, int aggr, int kernel,
                                         int64_t chunk, size_t *bytes);

/* pyg_propagate_edge with edge features of another width D (Eq. (1)'s
 * e_{j,i} in R^D): the features are first projected to F,
 * e = edge_attr Theta_e, by the dense transform (matrix cores, fp32
 * accumulation, e stored in dtype: rounded once for bf16), then propagated
 * as pyg_propagate_edge does with that e.
 *   edge_attr [E, D] in dtype and attr_order; theta_e [D, F] in dtype;
 *   everything else as pyg_propagate_edge. The projected features live in
 *   the workspace (E*F elements of dtype, then the two calls' workspaces).
 * Errors: as pyg_propagate_edge and pyg_dense_transform, plus
 * PYG_ERR_INVALID_ARG for NULL edge_attr or theta_e with E*D or D*F > 0 and
 * for x, edge_attr, theta_e or out overlapping the workspace. */
int pyg_propagate_edge_encoded(const void *x, int dtype, int64_t N, int64_t F, const int64_t *edge_index, int64_t E,
                               const void *edge_attr, int64_t D, const void *theta_e, int attr_order,
                               const pyg_csr *csr, int msg, int aggr, int kernel, void *out, int64_t *argmax,
                               void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_propagate_backward (chunk_t = csr_t->chunk). */
int pyg_propagate_backward_workspace(int dtype, int64_t N, int64_t F, int64_t E, int aggr, int64_t chunk_t,
                                     size_t *bytes);

/* Gradient of pyg_propagate for an upstream gradient g = dL/d out (the
 * backward pass that Appendix A compares for gather/scatter and SpMM):
 *   sum / mean (s_i = 1 or 1/deg_i):
 *     grad_x[j] = sum over edges k = (j -> i) of w_k s_i g_i, computed as a
 *     propagate over the transposed graph; difference messages
 *     (phi = x_j - x_i) add grad_x[i] -= deg_i s_i g_i;
 *     grad_w[k] = s_i <g_i, x_j> (weighted source messages only).
 *   max: each output element passes its gradient to its winning edge
 *     k = argmax[i,f]: grad_x[j,f] += w_k g_{i,f}, grad_w[k] += g_{i,f} x_{j,f};
 *     difference messages: grad_x[j,f] += g_{i,f}, grad_x[i,f] -= g_{i,f}.
 * Arguments:
 *   grad_out [N,F], x [N,F] (read only for grad_w), dtype of both;
 *   edge_index [2,E] COO (max only), edge_weight fp32 [E] COO order or NULL:
 *     the forward's weights; the call is weighted when it is non-NULL;
 *   csr    the forward CSR (rows = targets): required for mean, difference
 *          messages and grad_w (sum / mean);
 *   csr_t  the CSR of the reversed edge list (rows = sources), built by
 *          pyg_coo_to_csr from [edge_index[1]; edge_index[0]] with the same
 *          weights: required for sum / mean;
 *   argmax the forward's argmax [N,F] (max only);
 *   grad_x [N,F] output in dtype (fp32 accumulation);
 *   grad_w fp32 [E] output, or NULL to skip it, in w_order: PYG_ORDER_COO
 *          (edge ids, the order of edge_weight) or PYG_ORDER_CSR (the slots
 *          of csr, the order of csr->weight: coalesced stores, no scatter
 *          through perm); max in CSR order needs csr (with perm) too.
 * sum / mean results are deterministic; max scatters with float atomics, so
 * colliding winners may sum in any order (last-bit differences).
 * Errors: PYG_ERR_INVALID_ARG (bad dtype/msg/aggr/w_order, negative sizes,
 * NULL or mismatched CSRs or arrays that the call needs, grad_w without
 * weights, overlapping grad_x and inputs), PYG_ERR_UNSUPPORTED (N or
 * E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_propagate_backward(const void *grad_out, const void *x, int dtype, int64_t N, int64_t F,
                           const int64_t *edge_index, int64_t E, const float *edge_weight,
                           const pyg_csr *csr, const pyg_csr *csr_t, int msg, int aggr, const int64_t *argmax,
                           void *grad_x, float *grad_w, int w_order, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_propagate_edge_backward (chunk_t = csr_t->chunk
 * when grad_x is wanted under sum / mean, else 0). bf16 adds fp32 scratch:
 * N*F*4 bytes for grad_x under mean or max, and under mean with
 * max(x_j + e, 0) or x_j * e another N*F*4 + E*F*4 bytes (x and the edge
 * rows widened to fp32). Errors: PYG_ERR_INVALID_ARG (NULL bytes, negative
 * sizes, bad dtype/msg/aggr), PYG_ERR_UNSUPPORTED (N or E >= 2^31). */
int pyg_propagate_edge_backward_workspace(int dtype, int64_t N, int64_t F, int64_t E, int msg, int aggr,
                                          int64_t chunk_t, size_t *bytes);

/* Gradient of pyg_propagate_edge (Eq. (1) with F-dimensional edge features
 * e_{j,i}) for g = dL/d out [N, F]. Edge k = (j -> i) receives d_k = s_i g_i
 * (sum: s_i = 1, mean: 1/deg_i) or, for max, g_{i,f} in the columns f where
 * k = argmax[i, f]; through phi:
 *   x_j + e:          grad_x[j] += d_k,                 grad_e[k] = d_k;
 *   max(x_j + e, 0):  both times [x_j + e_k > 0];
 *   x_j * e:          grad_x[j] += d_k * e_k,           grad_e[k] = d_k * x_j.
 *   grad_out, x, edge_attr, grad_x, grad_edge_attr all in dtype (PYG_F32
 *     or PYG_BF16; bf16 is widened as it is loaded, every sum and product
 *     is fp32 and each gradient is rounded once); edge_attr and
 *     grad_edge_attr [E, F] in
 *     attr_order (PYG_ORDER_CSR: CSR slot order; PYG_ORDER_COO: edge id);
 *     x and edge_attr are not read for x_j + e (may be NULL there);
 *   csr     the forward's CSR (its E is the edge count); csr_t the CSR of
 *           the reversed edge list (sum / mean with grad_x); map_t its
 *           transpose map from pyg_csr_transpose_map (CSR order; NULL = made
 *           in the workspace); edge_index and argmax (the forward's) for max.
 *   Either output may be NULL, not both (unless both are empty).
 * sum / mean are deterministic; max adds into grad_x with float atomics.
 * Errors: PYG_ERR_INVALID_ARG (bad dtype/msg/aggr/order, negative sizes, NULL
 * or mismatched CSRs, missing arrays for the requested outputs),
 * PYG_ERR_UNSUPPORTED (N or E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_propagate_edge_backward(const void *grad_out, const void *x, const void *edge_attr, int dtype, int64_t N,
                                int64_t F, const int64_t *edge_index, const pyg_csr *csr, const pyg_csr *csr_t,
                                const int32_t *map_t, int attr_order, int msg, int aggr, const int64_t *argmax,
                                void *grad_x, void *grad_edge_attr, void *ws, size_t ws_bytes, void *stream);

/* ---- Attention (GAT, an operator of Section 2; Section 3, runtime
 * paragraph, credits its speed to a dedicated sparse softmax). Every edge
 * carries H fp32 values per array, row-major [E, H], in the order `order`
 * (pyg_order). The CSR fixes the segments: the incoming edges of each
 * target. Targets without incoming edges own no entries. All results are
 * bit-reproducible (fixed reduction orders). Sizes come from csr->N and
 * csr->E (E < 2^31); errors: PYG_ERR_INVALID_ARG for a NULL pointer that is
 * needed, H <= 0, an unknown order, or PYG_ORDER_COO without csr->perm. */

/* Workspace bytes needed by the three softmax calls below (same for all;
 * pass csr->chunk as chunk). */
int pyg_segment_softmax_workspace(int64_t E, int64_t N, int64_t H, int64_t chunk, size_t *bytes);

/* Softmax over the incoming edges of each target, per head h:
 *   alpha[k,h] = exp(s[k,h] - m[i,h]) / sum_{k' -> i} exp(s[k',h] - m[i,h]),
 *   m[i,h] = max_{k' -> i} s[k',h],  i = target of edge k.
 * scores and alpha fp32 [E, H] (device), may not overlap. fp32 arithmetic:
 * one online max/sum pass and one normalising pass.
 * Errors: PYG_ERR_INVALID_ARG (NULL or inconsistent csr, H <= 0, NULL
 * arrays, bad order, COO order without csr->perm), PYG_ERR_UNSUPPORTED (N or
 * E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_segment_softmax(const float *scores, int64_t H, const pyg_csr *csr, int order, float *alpha,
                        void *ws, size_t ws_bytes, void *stream);

/* GAT's attention coefficients in one call: the softmax above of the edge
 * scores e[k,h] = LeakyReLU(a_src[j,h] + a_dst[i,h]) for edge k = (j -> i),
 * LeakyReLU(v) = v for v >= 0 and negative_slope * v otherwise, computed on
 * the fly (never stored). a_src, a_dst fp32 [N, H] (device): the per-node
 * halves of GAT's attention vector applied to the transformed features.
 * Errors: as pyg_segment_softmax, plus PYG_ERR_INVALID_ARG for a
 * non-finite negative_slope. */
int pyg_gat_softmax(const float *a_src, const float *a_dst, int64_t H, float negative_slope, const pyg_csr *csr,
                    int order, float *alpha, void *ws, size_t ws_bytes, void *stream);

/* Gradient of the softmax with respect to its scores, for the upstream
 * gradient g = dL/d alpha:
 *   grad_scores[k,h] = alpha[k,h] * (g[k,h] - sum_{k' -> i} alpha[k',h] g[k',h]).
 * alpha, grad_alpha, grad_scores fp32 [E, H] (device); grad_scores may not
 * overlap the inputs.
 * Errors: as pyg_segment_softmax. */
int pyg_segment_softmax_backward(const float *alpha, const float *grad_alpha, int64_t H, const pyg_csr *csr,
                                 int order, float *grad_scores, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_propagate_heads (pass csr->chunk as chunk). */
int pyg_propagate_heads_workspace(int dtype, int64_t N, int64_t H, int64_t C, int64_t E, int64_t chunk,
                                  size_t *bytes);

/* Attention-weighted sum with H heads (GAT's message alpha_{j,i} x_j under
 * sum aggregation, Eq. (1), heads concatenated): x is [N, H*C] with head h
 * owning columns h*C .. h*C+C-1, and
 *   out[i, h*C + c] = sum over CSR slots p of row i of alpha[p,h] * x[col[p], h*C + c].
 *   x, out  [N, H*C] fp32 or bf16 (dtype), fp32 accumulation; rows take the
 *           16-byte vector path when C * sizeof(dtype) % 16 == 0;
 *   alpha   fp32 [E, H] in CSR slot order (PYG_ORDER_CSR); csr->weight is ignored.
 * Deterministic, same kernel and work split as pyg_propagate's CSR path.
 * Errors: PYG_ERR_INVALID_ARG (bad dtype, H <= 0, C < 0, NULL or
 * mismatched csr, NULL arrays, out overlapping x or alpha),
 * PYG_ERR_UNSUPPORTED (N, E or H*C >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_propagate_heads(const void *x, int dtype, int64_t N, int64_t H, int64_t C, const pyg_csr *csr,
                        const float *alpha, void *out, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_csr_transpose_map: E int32 of inverse
 * permutation, and from 2^20 edges on the scratch of its partition by edge
 * id (two 8-byte words and one byte per edge, plus digit counts).
 * Errors: PYG_ERR_INVALID_ARG (NULL bytes, E < 0), PYG_ERR_UNSUPPORTED
 * (E >= 2^31). */
int pyg_csr_transpose_map_workspace(int64_t E, size_t *bytes);

/* The transpose map between the CSR of an edge list (csr) and the CSR of
 * its reversed edge list (csr_t), both built by pyg_coo_to_csr:
 *   map_t[q] = the slot of csr that holds the edge of slot q of csr_t
 *              (the slot p with csr->perm[p] == csr_t->perm[q]).
 * int32 [E], caller-owned. Graph preprocessing like csr_t itself: made once
 * per graph, it lets the backward below read values kept in csr slot order
 * (the coefficients alpha, dL/dv) from the reversed CSR's rows without
 * re-ordering them. Entries of a malformed permutation are clamped into
 * [0, E) (results are then meaningless but every read stays in bounds).
 * Errors: PYG_ERR_INVALID_ARG (NULL or mismatched CSRs, no perm),
 * PYG_ERR_UNSUPPORTED (E >= 2^31), PYG_ERR_WORKSPACE. */
int pyg_csr_transpose_map(const pyg_csr *csr, const pyg_csr *csr_t, int32_t *map_t, void *ws, size_t ws_bytes,
                          void *stream);

/* Workspace bytes needed by pyg_propagate_heads_backward (pass csr_t->chunk). */
int pyg_propagate_heads_backward_workspace(int dtype, int64_t N, int64_t H, int64_t C, int64_t E, int64_t chunk_t,
                                           size_t *bytes);

/* Gradient of pyg_propagate_heads (GAT's attention sum, Eq. (1)) for
 * g = dL/d out [N, H*C]:
 *   grad_x[j, h*C + c]  = sum over edges k = (j -> i) of alpha[k,h] * g[i, h*C + c]
 *                         (the attention sum over the reversed graph; csr_t is
 *                         the CSR of the reversed edge list, built like csr);
 *   grad_alpha[p, h]    = sum_c g[row(p), h*C + c] * x[col[p], h*C + c], CSR
 *                         slot order of csr (the order of alpha).
 * grad_out, x, grad_x in dtype (fp32 accumulation); alpha, grad_alpha fp32
 * [E, H]. map_t: the transpose map of (csr, csr_t) from
 * pyg_csr_transpose_map, or NULL to make it in the workspace on every call.
 * Either output may be NULL (not both, unless both are empty); x is needed
 * for grad_alpha.
 * Deterministic. Errors: PYG_ERR_INVALID_ARG (NULL or mismatched CSRs,
 * missing arrays, H <= 0), PYG_ERR_UNSUPPORTED (N, E or H*C >= 2^31),
 * PYG_ERR_WORKSPACE. */
int pyg_propagate_heads_backward(const void *grad_out, const void *x, int dtype, int64_t N, int64_t H, int64_t C,
                                 const pyg_csr *csr, const pyg_csr *csr_t, const int32_t *map_t, const float *alpha,
                                 void *grad_x, float *grad_alpha, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_gat_scores_backward (pass csr_t->chunk). */
int pyg_gat_scores_backward_workspace(int64_t N, int64_t H, int64_t E, int64_t chunk_t, size_t *bytes);

/* Gradient of GAT's edge scores e = LeakyReLU(a_src[j] + a_dst[i]) for
 * g = dL/d e (fp32 [E, H], CSR slot order of csr, e.g. from
 * pyg_segment_softmax_backward with PYG_ORDER_CSR):
 *   dL/dv = g * (a_src[j,h] + a_dst[i,h] >= 0 ? 1 : negative_slope),
 *   grad_a_dst[i, h] = sum of dL/dv over the incoming edges of i,
 *   grad_a_src[j, h] = sum of dL/dv over the outgoing edges of j (rows of csr_t).
 * a_src, a_dst, grad_a_src, grad_a_dst fp32 [N, H]; map_t as for
 * pyg_propagate_heads_backward (or NULL). Deterministic. Errors as there,
 * plus PYG_ERR_INVALID_ARG for a non-finite negative_slope. */
int pyg_gat_scores_backward(const float *a_src, const float *a_dst, int64_t H, float negative_slope,
                            const pyg_csr *csr, const pyg_csr *csr_t, const int32_t *map_t, const float *grad_scores,
                            float *grad_a_src, float *grad_a_dst, void *ws, size_t ws_bytes, void *stream);

/* ---- Dense feature transform of a GCN layer (Section 2 lists GCN; its
 * layer multiplies the features by a weight matrix around the normalised
 * aggregation, A (X Theta) = (A X) Theta). */

/* Workspace bytes needed by pyg_dense_transform (Theta transposed and padded,
 * enough for either operand type). */
int pyg_dense_transform_workspace(int64_t Fi, int64_t Fo, size_t *bytes);

/* out[n, o] = sum_k x[n, k] * theta[k, o] on the matrix cores, fp32
 * accumulation: bf16 operands (exact products, v_mfma_f32_16x16x32_bf16) or
 * fp32 operands (v_mfma_f32_16x16x4_f32).
 *   x      [N, Fi] in x_dtype (PYG_BF16 or PYG_F32); 16-byte aligned rows
 *          (Fi % 8 == 0 for bf16, Fi % 4 == 0 for fp32) take the vector path;
 *   theta  [Fi, Fo] row-major, in x_dtype;
 *   out    [N, Fo] in out_dtype (PYG_F32, or PYG_BF16 rounded once), may not
 *          overlap x.
 * Deterministic. Errors: PYG_ERR_INVALID_ARG (bad dtypes, NULL pointers,
 * negative sizes, overlap), PYG_ERR_UNSUPPORTED (N >= 2^31, Fi or Fo >=
 * 2^24), PYG_ERR_WORKSPACE. */
int pyg_dense_transform(const void *x, int x_dtype, int64_t N, int64_t Fi, const void *theta, int64_t Fo,
                        void *out, int out_dtype, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes needed by pyg_global_pool. */
int pyg_global_pool_workspace(int dtype, int64_t N, int64_t F, int64_t B, int aggr, size_t *bytes);

/* Global pooling (Section 2, "Global Pooling" with the assignment vector of
 * "Mini-batch Handling"): out[g, f] = AGG over nodes n with batch[n] = g of
 * x[n, f], for B graphs.
 *   batch int64 [N], non-decreasing, values in [0, B);
 *   out   [B,F] in x's dtype; argmax int64 [B,F] (PYG_MAX only): node id,
 *         N for an empty graph.
 * Errors: PYG_ERR_INVALID_ARG (bad dtype/aggr, negative sizes, NULL
 * arrays, argmax given without max or missing with it, B = 0 with nodes,
 * out overlapping x), PYG_ERR_UNSUPPORTED (N or B >= 2^31),
 * PYG_ERR_WORKSPACE. */
int pyg_global_pool(const void *x, int dtype, int64_t N, int64_t F, const int64_t *batch, int64_t B,
                    int aggr, void *out, int64_t *argmax, void *ws, size_t ws_bytes, void *stream);

/* Count COO entries outside [0, N) into *bad_count (int64, device).
 * Errors: PYG_ERR_INVALID_ARG (negative sizes, NULL bad_count or
 * edge_index). */
int pyg_validate_coo(const int64_t *edge_index, int64_t E, int64_t N, int64_t *bad_count, void *stream);

/* Count batch entries outside [0, B) or smaller than their predecessor into
 * *bad_count (int64, device).
 * Errors: PYG_ERR_INVALID_ARG (negative sizes, NULL bad_count or batch). */
int pyg_validate_batch(const int64_t *batch, int64_t N, int64_t B, int64_t *bad_count, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PYG_MI355X_H */
