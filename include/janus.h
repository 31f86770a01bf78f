/*
 * janus.h - C ABI of the MI355X (gfx950) training-step library.
 *
 * The library runs one whole training step (forward and backward) of a
 * dynamic-control-flow model on the GPU: an LSTM driven by a loop whose trip
 * count depends on the data (per-sequence lengths), and a binary TreeLSTM
 * driven by recursion over trees, evaluated level by level.  These are the
 * loops and recursive calls of the paper's imperative programs (Figure 1;
 * Section 4.2.1, dynamic control flow), executed as one device program per
 * call instead of per-operation dispatch.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Tensors are caller-owned DEVICE pointers, dense, row-major, with the
 *    shapes given below.  "dtype" tensors hold float32 or bf16 (raw 16-bit
 *    patterns) as selected by the descriptor; float* tensors are always
 *    float32.  Gradients are float32 and are OVERWRITTEN, never accumulated.
 *  - Arrays documented as "host" are read during the call only.
 *  - Each call enqueues its kernels on `stream` (a hipStream_t, 0 = the null
 *    stream) and returns without synchronising; device faults surface at the
 *    caller's next synchronisation.  Calls are re-entrant given distinct
 *    workspaces.
 *  - Workspaces are caller-allocated device memory of at least the size
 *    returned by the matching *_workspace_bytes function, 256-byte aligned.
 *    The forward call stores the values its backward needs there; the
 *    workspace must not be modified between a forward call and its backward.
 *    The library allocates no device memory.
 *  - All validation happens before the first device operation.  When a call
 *    returns anything other than JANUS_OK before launching, no output buffer
 *    has been written (all-or-nothing state updates, Section 3.2 and
 *    Section 4.2.3).  JANUS_ERR_DEVICE means a HIP call failed after work was
 *    enqueued; outputs are then undefined.
 */
#ifndef JANUS_H
#define JANUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    JANUS_OK = 0,
    JANUS_ERR_INVALID_ARG = 1,   /* NULL required pointer, non-positive size   */
    JANUS_ERR_LENGTH = 2,        /* sequence length outside [0, T]             */
    JANUS_ERR_TREE = 3,          /* malformed tree batch                       */
    JANUS_ERR_TOKEN = 4,         /* token / word / class id outside [0, V)     */
    JANUS_ERR_WORKSPACE = 5,     /* workspace missing, too small or misaligned */
    JANUS_ERR_UNSUPPORTED = 6,   /* dtype or shape combination not built       */
    JANUS_ERR_DEVICE = 7         /* a HIP call failed                          */
} janus_status;

typedef enum { JANUS_F32 = 0, JANUS_BF16 = 1 } janus_dtype;

/* ------------------------------------------------------------------------ */
/* LSTM over variable-length sequences                                      */
/* ------------------------------------------------------------------------ */

/* L stacked layers, input size I, hidden size H, batch B, T time steps. */
typedef struct {
    int32_t L, I, H, B, T;
    janus_dtype dtype;
} janus_lstm_desc;

/* Bytes of workspace needed by janus_lstm_seq_fwd / _bwd for this shape. */
size_t janus_lstm_workspace_bytes(const janus_lstm_desc* d);

/*
 * Forward pass of the recurrence of Figure 1 (``state = rnn_cell(state,
 * item)`` for every item), with the standard LSTM cell of the LSTM / LM
 * models of Section 6.1:
 *     a = Wx x_t + Wh h_{t-1} + b   (gate blocks i, f, g, o)
 *     c_t = s(a_f) c_{t-1} + s(a_i) tanh(a_g),   h_t = s(a_o) tanh(c_t)
 * Sequence b advances while t < lengths[b] (a loop with a data-dependent
 * trip count, Section 4.2.1); afterwards its state is carried unchanged and
 * its output is 0.  Layer l+1 reads the output of layer l.
 *
 *  x        [T, B, I] dtype, time-major.
 *  lengths  host int32 [B] with 0 <= len <= T, or NULL for all T.
 *  Wx[l]    [4H, I_l] dtype (I_0 = I, I_l = H above), Wh[l] [4H, H] dtype,
 *  b[l]     [4H] dtype: host arrays of L device pointers, the per-layer
 *           layout of torch.nn.LSTM weight_ih_l{k} / weight_hh_l{k} with one
 *           bias.
 *  h0, c0   [L, B, H] float32 or NULL (zeros).
 *  y        [T, B, H] dtype: top-layer output; 0 where t >= len_b.
 *  hT, cT   [L, B, H] float32 or NULL: state after len_b steps (= h0, c0 for
 *           a length-0 sequence).
 *  ws       workspace (see conventions); the forward keeps activations there.
 *
 * Errors: NULL d/Wx/Wh/b/ws, NULL x or y with T > 0, a non-positive L, I, H, B, or T < 0
 * -> INVALID_ARG; a length outside [0, T] -> LENGTH; ws_bytes too small ->
 * WORKSPACE; dtype not F32/BF16 -> UNSUPPORTED.
 */
janus_status janus_lstm_seq_fwd(const janus_lstm_desc* d, const void* x,
                                const int32_t* lengths,
                                const void* const* Wx, const void* const* Wh,
                                const void* const* b,
                                const float* h0, const float* c0,
                                void* y, float* hT, float* cT,
                                void* ws, size_t ws_bytes, void* stream);

/*
 * Backward pass through time of the call above (same d, x, lengths, Wx,
 * Wh and the workspace it filled).
 *
 *  dy       [T, B, H] dtype gradient of y, or NULL (zero).  Entries where
 *           t >= len_b are ignored (y is the constant 0 there).
 *  dhT, dcT [L, B, H] float32 or NULL (zero).
 *  dx       [T, B, I] dtype gradient of x, or NULL to skip it; 0 where
 *           t >= len_b.
 *  dh0, dc0 [L, B, H] float32 or NULL.
 *  dWx[l], dWh[l], db[l]: host arrays of L device float32 pointers with the
 *           shapes of Wx[l], Wh[l], b[l].
 * Errors as for the forward call; additionally NULL dWx/dWh/db.
 */
janus_status janus_lstm_seq_bwd(const janus_lstm_desc* d, const void* x,
                                const int32_t* lengths,
                                const void* const* Wx, const void* const* Wh,
                                void* ws, size_t ws_bytes,
                                const void* dy, const float* dhT, const float* dcT,
                                void* dx, float* dh0, float* dc0,
                                float* const* dWx, float* const* dWh, float* const* db,
                                void* stream);

/*
 * Carries the recurrent state of one batch into the next: the program of
 * Figure 1 keeps the state in self.state between calls, and the stored
 * state changes only after a whole step has run (deferred state update,
 * Section 4.2.3), so this call belongs after the step's backward call.
 *  d        descriptor of the NEXT batch (L, H, B = B_next; I, T unused but
 *           validated as for the other calls).
 *  B_prev   rows of the previous batch, >= 0 (0: no previous batch).
 *  hT, cT   [L, B_prev, H] float32: final state of the previous batch (may be
 *           NULL when B_prev is 0).
 *  h0, c0   [L, B_next, H] float32, written: row r of layer l continues
 *           (= hT, cT) for r < B_prev, starts from 0 otherwise; rows
 *           r >= B_next of the previous batch end (a smaller last batch).
 * Errors: bad d -> as janus_lstm_seq_fwd; B_prev < 0, NULL h0/c0, NULL
 * hT/cT with B_prev > 0, or any of the four buffers overlapping another ->
 * INVALID_ARG.
 */
janus_status janus_lstm_state_carry(const janus_lstm_desc* d, int32_t B_prev,
                                    const float* hT, const float* cT,
                                    float* h0, float* c0, void* stream);

/*
 * Report of the current step made with this workspace (same d): the last
 * janus_lstm_seq_fwd call and the janus_lstm_seq_bwd calls after it.  The
 * persistent recurrence kernels separate their time steps with device-wide
 * barriers whose waits are bounded; when a wait runs out, the kernels drain
 * and the outputs are undefined.  Those calls return without synchronising,
 * so this call synchronises `stream` and reads the report back.  Reading does
 * not clear it; the next forward call does.
 *  timed_out         1 if any wait of the step ran out (forward or
 *                    backward: the backward keeps the forward's flag, and
 *                    its kernels then drain at once).
 *  bwd_groups        backward unit groups launched by the last backward
 *                    call, summed over layers (0 when the per-step kernels
 *                    ran, or before a backward).
 *  bwd_local_groups  of those, groups whose workgroups all ran on one XCD
 *                    and kept their partial sums in its L2.
 *  fwd_groups, fwd_local_groups  the same for the forward recurrence when
 *                    its contraction is split over the columns of Wh (0
 *                    otherwise).
 * Errors: INVALID_ARG (bad d, NULL out), WORKSPACE (as for the calls above),
 * DEVICE (a HIP call failed, or timed_out is 1).
 */
typedef struct {
    int32_t timed_out;
    int32_t bwd_groups;
    int32_t bwd_local_groups;
    int32_t fwd_groups;
    int32_t fwd_local_groups;
} janus_lstm_report;

janus_status janus_lstm_device_report(const janus_lstm_desc* d, const void* ws, size_t ws_bytes,
                                      janus_lstm_report* out, void* stream);

/*
 * Device address of the timeout flag inside an LSTM workspace (no device
 * work, no synchronisation).  The word is a uint32 that janus_lstm_seq_fwd
 * clears when it starts and that the persistent kernels set when a bounded
 * wait runs out; janus_lstm_seq_bwd leaves it as it is, so after a step it is
 * non-zero if any wait of the step's forward or backward ran out.  Hand it to
 * janus_sgd_clip_update as `hold` to keep a failed step from updating the
 * parameters (state changes are all-or-nothing, Section 4.2.3).  The address
 * stays valid as long as the workspace does.
 * Errors: INVALID_ARG (bad d, NULL out), WORKSPACE (as for the calls above).
 */
janus_status janus_lstm_fault_flag(const janus_lstm_desc* d, const void* ws, size_t ws_bytes,
                                   const uint32_t** out);

/*
 * Integer schedule of the sequence loop (host only, no device use):
 *  perm[B]       batch indices sorted by (-len_b, b)
 *  active[T]     active[t] = #{b : len_b > t} for t < t_eff, 0 after
 *  offsets[T+1]  offsets[t] = sum of active[t'] for t' < t
 *  t_eff         max len (the loop's trip count)
 * Errors: INVALID_ARG for NULL pointers or B <= 0, T < 0; LENGTH.
 */
janus_status janus_lstm_schedule(int32_t B, int32_t T, const int32_t* lengths,
                                 int32_t* perm, int32_t* active, int32_t* offsets,
                                 int32_t* t_eff);

/* ------------------------------------------------------------------------ */
/* Binary TreeLSTM over a batch of trees                                    */
/* ------------------------------------------------------------------------ */

/* Embedding size E, hidden size H, vocabulary V. */
typedef struct {
    int32_t E, H, V;
    janus_dtype dtype;
} janus_treelstm_desc;

/*
 * A batch of binary trees as HOST int32 arrays of num_nodes entries:
 * left[n], right[n] are child node ids, both -1 for a leaf; word[n] is the
 * token id of a leaf (in [0, V)) and -1 for an internal node.  root[k]
 * (num_trees entries) is the root of tree k.  Every node has at most one
 * parent and is reachable from exactly one root.  Node order is arbitrary.
 */
typedef struct {
    int32_t num_trees, num_nodes;
    const int32_t* left;
    const int32_t* right;
    const int32_t* word;
    const int32_t* root;
} janus_tree_batch;

/* Workspace bytes for a batch of at most max_nodes nodes and max_trees trees. */
size_t janus_treelstm_workspace_bytes(const janus_treelstm_desc* d, int32_t max_nodes,
                                      int32_t max_trees);

/*
 * Frontier schedule of the recursion (host only): level(leaf) = 0,
 * level(n) = 1 + max(level(left), level(right)); level_nodes lists node
 * ids sorted by (level, id); level_offsets[k] = #{n : level(n) < k}.
 *  node_level[num_nodes], level_offsets[num_nodes + 1], level_nodes[num_nodes].
 * Errors: INVALID_ARG (NULL, empty batch), TREE (one child, two parents,
 * bad id, cycle, unreachable node, internal node with a word), TOKEN (leaf
 * word outside [0, V)).
 */
janus_status janus_tree_schedule_build(const janus_tree_batch* t, int32_t V,
                                       int32_t* node_level, int32_t* level_offsets,
                                       int32_t* level_nodes, int32_t* num_levels);

/*
 * Forward pass of the recursive TreeNN program (Section 6.1, footnote 6;
 * recursion as graph invocations, Section 4.2.1), evaluated one level of
 * independent nodes at a time.  Cell of node n (binary TreeLSTM of the SST
 * model, Table 2):
 *     a = b + (leaf ? W emb[word[n]] : U [h_L; h_R])
 *     gate blocks (i, f_L, f_R, o, u); c = s(i) tanh(u) + s(f_L) c_L + s(f_R) c_R
 *     h = s(o) tanh(c); leaves have zero children.
 *  emb [V, E], W [5H, E], U [5H, 2H], b [5H]: dtype.
 *  h_root [num_trees, H] dtype: h of root[k].
 * Errors: INVALID_ARG, TREE, TOKEN, WORKSPACE, UNSUPPORTED (only F32).
 */
janus_status janus_treelstm_fwd(const janus_treelstm_desc* d, const janus_tree_batch* t,
                                const void* emb, const void* W, const void* U,
                                const void* b, void* h_root,
                                void* ws, size_t ws_bytes, void* stream);

/*
 * Backward of the call above (same d, t, emb, W, U and workspace; the
 * workspace must be left unchanged between the two calls: it holds the
 * forward's gates, cells and uploaded schedule).
 *  dh_root [num_trees, H] dtype: gradient of h_root (gradient of the roots'
 *          c is zero).
 *  demb [V, E], dW [5H, E], dU [5H, 2H], db [5H]: float32, overwritten
 *          (rows of demb for words not in the batch are 0).
 * Where the weight slices fit one CU's LDS each direction is one launch of
 * co-resident workgroups that runs every level with a device-wide barrier
 * between levels (the waits are bounded; see janus_treelstm_device_report).
 */
janus_status janus_treelstm_bwd(const janus_treelstm_desc* d, const janus_tree_batch* t,
                                const void* emb, const void* W, const void* U,
                                void* ws, size_t ws_bytes, const void* dh_root,
                                float* demb, float* dW, float* dU, float* db,
                                void* stream);

/*
 * Device-side status of the TreeLSTM calls made with this workspace since
 * the last forward (same d and t).  Synchronises `stream`, then sets
 * *timed_out = 1 if a level barrier of the forward or backward ran out of
 * its bounded wait (their results are then undefined) and returns
 * JANUS_ERR_DEVICE; else *timed_out = 0 and JANUS_OK.  The flag is cleared
 * by the next forward.  Errors: as janus_treelstm_fwd's validation, or
 * INVALID_ARG for a NULL timed_out.
 */
janus_status janus_treelstm_device_report(const janus_treelstm_desc* d, const janus_tree_batch* t,
                                          const void* ws, size_t ws_bytes, int32_t* timed_out,
                                          void* stream);

/* ------------------------------------------------------------------------ */
/* Binary TreeRNN over a batch of trees                                     */
/* ------------------------------------------------------------------------ */

/*
 * The paper's other TreeNN (TreeRNN on SST, Table 2), on the same frontier
 * schedule and tree batches as the TreeLSTM.  Cell of node n:
 *     h = emb[word[n]]                      (leaf: its word vector)
 *     h = tanh(W [h_L; h_R] + b)            (internal node)
 * The descriptor is the TreeLSTM's with E = H (the leaf h is the embedding).
 */
typedef janus_treelstm_desc janus_treernn_desc;

/* Workspace bytes for a batch of at most max_nodes nodes and max_trees
 * trees (0 for a bad descriptor, including E != H). */
size_t janus_treernn_workspace_bytes(const janus_treernn_desc* d, int32_t max_nodes,
                                     int32_t max_trees);

/*
 *  emb [V, H], W [H, 2H], b [H]: float32.
 *  h_root [num_trees, H] float32: h of root[k].
 * Errors: INVALID_ARG (as for the TreeLSTM, or E != H), TREE, TOKEN,
 * WORKSPACE, UNSUPPORTED (only F32).
 */
janus_status janus_treernn_fwd(const janus_treernn_desc* d, const janus_tree_batch* t,
                               const void* emb, const void* W, const void* b,
                               void* h_root, void* ws, size_t ws_bytes, void* stream);

/*
 * Backward of the call above (same d, t, W and workspace).
 *  dh_root [num_trees, H] float32: gradient of h_root.
 *  demb [V, H], dW [H, 2H], db [H]: float32, overwritten (rows of demb for
 *          words not in the batch are 0; a leaf's gradient is its dh).
 * Errors: as the forward.
 */
janus_status janus_treernn_bwd(const janus_treernn_desc* d, const janus_tree_batch* t,
                               const void* W, void* ws, size_t ws_bytes,
                               const void* dh_root, float* demb, float* dW, float* db,
                               void* stream);

/*
 * Device-side status of the TreeRNN calls made with this workspace since the
 * last forward (same d and t), as janus_treelstm_device_report: where the
 * weight slices fit one CU's LDS (H up to about 312) each direction is one
 * launch of co-resident workgroups with a device-wide barrier between levels
 * (Section 4.2.1 recursion, run level by level); a barrier that ran out of
 * its bounded wait sets *timed_out = 1 and the call returns
 * JANUS_ERR_DEVICE (the results are then undefined).  The flag is cleared by
 * the next forward.  Errors: as janus_treernn_fwd's validation, or
 * INVALID_ARG for a NULL timed_out.
 */
janus_status janus_treernn_device_report(const janus_treernn_desc* d, const janus_tree_batch* t,
                                         const void* ws, size_t ws_bytes, int32_t* timed_out,
                                         void* stream);

/* ------------------------------------------------------------------------ */
/* Child-Sum TreeLSTM over trees of any arity                               */
/* ------------------------------------------------------------------------ */

/*
 * The other variant of the TreeLSTM the paper trains ([40]): nodes may have
 * any number of children and every node reads its word vector x.  With h~
 * the sum of the children's h:
 *     i = s(W_i x + U_i h~ + b_i),  o = s(W_o x + U_o h~ + b_o),
 *     u = tanh(W_u x + U_u h~ + b_u),  f_k = s(W_f x + U_f h_k + b_f) per child,
 *     c = i u + sum_k f_k c_k,  h = o tanh(c).
 * Gate blocks of W [4H, E], U [4H, H], b [4H] are (i, o, u, f).  Evaluated
 * one level of independent nodes at a time, as the binary TreeNNs.
 */
typedef janus_treelstm_desc janus_childsum_desc;

/*
 * A batch of trees as HOST int32 arrays: the children of node n are
 * children[child_offsets[n] .. child_offsets[n + 1]) (none: a leaf);
 * child_offsets has num_nodes + 1 entries starting at 0; word[n] in [0, V)
 * for every node; root[k] (num_trees entries) is the root of tree k.  Every
 * node has at most one parent and is reachable from exactly one root.
 */
typedef struct {
    int32_t num_trees, num_nodes;
    const int32_t* child_offsets;
    const int32_t* children;
    const int32_t* word;
    const int32_t* root;
} janus_nary_tree_batch;

/* Workspace bytes for a batch of at most max_nodes nodes. */
size_t janus_childsum_workspace_bytes(const janus_childsum_desc* d, int32_t max_nodes);

/*
 *  emb [V, E], W [4H, E], U [4H, H], b [4H]: float32.
 *  h_root [num_trees, H] float32: h of root[k].
 * Errors: INVALID_ARG (NULL pointers or arrays, empty batch, a non-positive
 * size), TREE (offsets not starting at 0 or decreasing, a child id out of
 * range, a node with two parents, a root with a parent, a cycle, a node no
 * root reaches), TOKEN (a word outside [0, V)), WORKSPACE, UNSUPPORTED (only
 * F32).
 */
janus_status janus_childsum_fwd(const janus_childsum_desc* d, const janus_nary_tree_batch* t,
                                const void* emb, const void* W, const void* U, const void* b,
                                void* h_root, void* ws, size_t ws_bytes, void* stream);

/*
 * Backward of the call above (same d, t, emb, W, U and workspace).
 *  dh_root [num_trees, H] float32: gradient of h_root (the roots' c gets 0).
 *  demb [V, E], dW [4H, E], dU [4H, H], db [4H]: float32, overwritten (rows
 *          of demb for words not in the batch are 0).
 * Errors: as the forward.
 */
janus_status janus_childsum_bwd(const janus_childsum_desc* d, const janus_nary_tree_batch* t,
                                const void* emb, const void* W, const void* U,
                                void* ws, size_t ws_bytes, const void* dh_root,
                                float* demb, float* dW, float* dU, float* db, void* stream);

/*
 * Device-side status of the Child-Sum calls made with this workspace since
 * the last forward (same d and t), as janus_treelstm_device_report: where
 * the weight slices fit one CU's LDS (H up to about 156, E up to 512) each
 * direction is one launch of co-resident workgroups with device-wide
 * barriers between levels (Section 4.2.1 recursion, run level by level); a
 * barrier that ran out of its bounded wait sets *timed_out = 1 and the call
 * returns JANUS_ERR_DEVICE (the results are then undefined).  The flag is
 * cleared by the next forward.  Errors: as janus_childsum_fwd's validation,
 * or INVALID_ARG for a NULL timed_out.
 */
janus_status janus_childsum_device_report(const janus_childsum_desc* d, const janus_nary_tree_batch* t,
                                          const void* ws, size_t ws_bytes, int32_t* timed_out,
                                          void* stream);

/* ------------------------------------------------------------------------ */
/* Embedding and softmax cross-entropy                                      */
/* ------------------------------------------------------------------------ */

typedef enum {
    JANUS_EMBED_FWD = 0,     /* out[r, :] = table[ids[r], :]                         */
    JANUS_XENT_FWD_BWD = 1,  /* mean cross-entropy of h table^T + bias, all grads   */
    JANUS_EMBED_BWD = 2      /* dtable[v, :] = sum of in[r, :] over ids[r] == v     */
} janus_xent_op;

/* Vocabulary (or class count) V, row width H, number of rows. */
typedef struct {
    int32_t V, H, rows;
    janus_dtype dtype;
} janus_xent_desc;

size_t janus_xent_workspace_bytes(const janus_xent_desc* d, janus_xent_op op);

/*
 * One of three operations around the LSTM language model and the tree root
 * classifier (the loss computed at the end of the Figure 1 program):
 *  ids_host [rows] host int32 and ids_dev [rows] device int32: the same
 *           ids (token ids for EMBED_*, target classes for XENT).
 *  EMBED_FWD:  table = E [V, H] dtype; out = x [rows, H] dtype.
 *  XENT_FWD_BWD: table = Wout [V, H], bias = bout [V], in = h [rows, H]
 *           (dtype); loss (device float32 scalar) = mean over rows of
 *           -log softmax(h Wout^T + bout)[ids[r]]; out = dh [rows, H] dtype;
 *           dtable = dWout [V, H], dbias = dbout [V] float32.
 *  EMBED_BWD:  in = dx [rows, H] dtype; dtable = dE [V, H] float32
 *           (deterministic: each row of dE sums its rows in ascending r;
 *           rows of ids not present are 0).  The rows are grouped by id on
 *           the host from ids_host (a stable counting sort, O(rows + V)) and
 *           one workgroup sums each group; any number of rows.
 *  ws:      XENT_FWD_BWD and EMBED_BWD take a workspace of
 *           janus_xent_workspace_bytes(d, op) bytes (256-byte aligned; for
 *           EMBED_BWD 12 bytes per row); EMBED_FWD takes none (NULL).
 * Errors: INVALID_ARG, TOKEN (an id outside [0, V)), WORKSPACE.
 */
janus_status janus_embed_softmax_xent(const janus_xent_desc* d, janus_xent_op op,
                                      const int32_t* ids_host, const int32_t* ids_dev,
                                      const void* table, const void* bias,
                                      const void* in, void* out,
                                      float* dtable, float* dbias, float* loss,
                                      void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------------ */
/* Regression head and scalar losses                                        */
/* ------------------------------------------------------------------------ */

typedef struct {
    int32_t rows, H, P;
    janus_dtype dtype;
} janus_mse_desc;

size_t janus_mse_workspace_bytes(const janus_mse_desc* d);

/*
 * Per-row linear projection and mean-squared error:
 *   yp = h W^T + b,  loss = mean over rows*P of (yp - target)^2
 *  h [rows, H], W [P, H], b [P], target [rows, P]: dtype.
 *  dh [rows, H] dtype; dW [P, H], db [P] float32; loss device float32.
 */
janus_status janus_linear_mse(const janus_mse_desc* d, const void* h, const void* W,
                              const void* b, const void* target, void* dh,
                              float* dW, float* db, float* loss,
                              void* ws, size_t ws_bytes, void* stream);

typedef enum {
    JANUS_LOSS_SUMSQ = 0,    /* loss = sum h^2,   dh = 2 h   */
    JANUS_LOSS_MEAN = 1      /* loss = mean h,    dh = 1 / n */
} janus_loss_kind;

/* h [n] float32 device; loss device float32 scalar; dh [n] float32 or NULL. */
janus_status janus_loss_reduce(janus_loss_kind kind, const float* h, int64_t n,
                               float* loss, float* dh, void* stream);

/* ------------------------------------------------------------------------ */
/* Tracing                                                                  */
/* ------------------------------------------------------------------------ */

/*
 * Per-kernel timing of the library's own launches.  Between
 * janus_trace_begin and janus_trace_end every kernel the library enqueues is
 * bracketed by two HIP events recorded on the stream it is launched on.
 * janus_trace_end waits for those events and returns one record per kernel
 * label, in order of first launch: the launch count, the summed event time
 * and the summed algorithmic work of the launches (2*M*N*K flops for a
 * contraction, bytes a kernel must move at minimum for memory-bound ones).
 * Tracing adds two event records per launch; it is meant for measurement
 * runs, not for the timed loop.  Not thread-safe against concurrent calls
 * from other threads.
 *  out: caller array of max_out records; n_out receives the number of labels
 *  (records beyond max_out are dropped).
 * Errors: INVALID_ARG (NULL n_out), DEVICE (an event call failed).
 */
typedef struct {
    char label[48];
    int64_t launches;
    double total_ms;
    double flops;
    double bytes;
} janus_trace_stat;

janus_status janus_trace_begin(void);
janus_status janus_trace_end(janus_trace_stat* out, int32_t max_out, int32_t* n_out);

/* ------------------------------------------------------------------------ */
/* Parameter update                                                         */
/* ------------------------------------------------------------------------ */
/*
 * SGD with the step scaled down by the global L2 norm of the gradients.  The
 * paper inserts the parameter update into the generated graph after the
 * gradients (Section 3.1) and names no optimizer; the rule here is
 *   norm = sqrt(sum over all tensors and entries of g^2),
 *   s    = min(1, max_norm / (norm + 1e-6)), or 1 when max_norm <= 0 or +inf,
 *   p   <- p - lr * s * g            (computed in float32, stored as dtype).
 * State changes are all-or-nothing (Section 4.2.3): when the norm is not
 * finite (a NaN or infinite gradient) no parameter is written.  The norm is
 * summed in float64 in a fixed order, so repeated calls give the same result.
 */
typedef struct {
    int32_t n;            /* parameter tensors, >= 1 */
    janus_dtype dtype;    /* of the parameters, F32 or BF16 (gradients are float32) */
    float lr;             /* learning rate, finite */
    float max_norm;       /* clipping threshold; <= 0 or +inf turns clipping off; not NaN */
} janus_sgd_desc;

/* Workspace bytes for janus_sgd_clip_update with this descriptor (0 for a
 * bad descriptor). */
size_t janus_sgd_workspace_bytes(const janus_sgd_desc* d);

/*
 *  params[i] host array of n device pointers to the parameters (dtype),
 *            updated in place; grads[i] host array of n device pointers to
 *            their float32 gradients; sizes[i] host array of n element
 *            counts (>= 0; a tensor of 0 elements may have NULL pointers).
 *            Tensors are flat and contiguous; parameters and gradients must
 *            not overlap.
 *  stats     device float32[2] or NULL: [0] the norm before clipping, [1]
 *            the scale s applied (0 when the update was skipped).
 *  hold      device uint32 or NULL.  Read when the update runs (stream
 *            order): if it is non-zero, no parameter is written, as for a
 *            non-finite norm.  Pass janus_lstm_fault_flag's word so that a
 *            training step whose recurrence timed out leaves the parameters
 *            unchanged (all-or-nothing, Section 4.2.3).
 *  ws        workspace (see conventions), at least
 *            janus_sgd_workspace_bytes(d) bytes.
 * Errors: NULL d/params/grads/sizes, n < 1, non-finite lr, NaN max_norm, a
 * negative size, a NULL pointer of a non-empty tensor, or a pointer not
 * aligned to its element -> INVALID_ARG; dtype not F32/BF16 -> UNSUPPORTED;
 * ws missing, too small or misaligned -> WORKSPACE.
 */
janus_status janus_sgd_clip_update(const janus_sgd_desc* d, void* const* params,
                                   const float* const* grads, const int64_t* sizes,
                                   float* stats, const uint32_t* hold, void* ws, size_t ws_bytes,
                                   void* stream);

/*
 * janus_sgd_clip_update for callers that cannot allocate device memory:
 * code under stream capture, tight serving loops, harnesses that forbid
 * hipMalloc.  Same arguments, rule and results as janus_sgd_clip_update,
 * without ws / ws_bytes: the block sums of the norm and the control word live
 * in a fixed array of the library (one per device, 33 KB, room for
 * JANUS_SGD_NOALLOC_MAX_TENSORS tensors), whose device address the library
 * looks up at the first call on each device and keeps until the process
 * ends.  The call allocates nothing (no hipMalloc, no events, no tracing).
 * Every call on one device shares that device's array: calls that overlap
 * on one device (several streams or host threads) race, and the caller must
 * order them.  Each call writes everything in the array that it reads, so
 * nothing carries over from the previous call.
 * Errors: as janus_sgd_clip_update (bad arguments -> INVALID_ARG, dtype ->
 * UNSUPPORTED); n > JANUS_SGD_NOALLOC_MAX_TENSORS -> WORKSPACE; a failed
 * lookup of the array -> DEVICE.
 */
#define JANUS_SGD_NOALLOC_MAX_TENSORS 256
janus_status janus_sgd_clip_update_noalloc(const janus_sgd_desc* d, void* const* params,
                                           const float* const* grads, const int64_t* sizes,
                                           float* stats, const uint32_t* hold, void* stream);

/* ------------------------------------------------------------------------ */
/* Misc                                                                     */
/* ------------------------------------------------------------------------ */
const char* janus_status_string(janus_status s);
const char* janus_version(void);
/* Text naming the HIP call behind the last JANUS_ERR_DEVICE returned on the
 * calling thread (HIP error name and code, the call, source file and line),
 * or "" before any.  The string is owned by the library and stays valid until
 * the next such error on the thread. */
const char* janus_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* JANUS_H */
