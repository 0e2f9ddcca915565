/*
 * tgm.h -- C ABI of libtgm, the MI355X (gfx950) implementation of the per-batch
 * memory-module stage of memory-based temporal GNN training.
 *
 * Method: MSPipe, "Efficient Temporal GNN Training via Staleness-Aware
 * Pipeline" (Sheng, Su, Huang, Wu; KDD'24, arXiv 2402.15113).  One training
 * iteration i processes a batch of B consecutive events of a time-sorted event
 * stream (Sec. 2, event-based dynamic graphs).  Its memory-module stage is:
 *
 *   tgm_batch_roots    roots of the batch: sources, destinations, negatives
 *   tgm_sample         most-recent-nb temporal neighbours of every root
 *   tgm_node_set       sorted unique node set U of roots and neighbours
 *   tgm_fetch_memory   node memory and mailbox of U as of iteration i-1-s
 *   tgm_update_memory  GRU memory update of U, latest-message reduce,
 *                      staged write-back of the batch's endpoints
 *   tgm_embed          time-encoded multi-head attention embedding of roots
 *   tgm_stage_run      all of it for a range of iterations, sampling a chunk
 *                      of iterations ahead on a second stream
 *
 * Conventions shared by every call:
 *  - All array arguments are DEVICE pointers unless marked "host".  Arrays are
 *    dense and row-major; "[a x b]" means a rows of b elements.
 *  - Ids are int32 in [0, N); timestamps are fp64; features, memory and
 *    weights are fp32.  Event e (0-based) has src[e], dst[e], t[e], neg[e] and
 *    edge-feature row efeat[e].  Events are sorted by (t, e).
 *  - Every compute call takes a HIP stream (hipStream_t passed as void*; NULL
 *    is the legacy default stream), enqueues its kernels there and returns
 *    without synchronising.  Argument checks are done on the host before
 *    anything is enqueued; on failure nothing is enqueued.  Faults raised by
 *    the device surface after the caller synchronises, through
 *    tgm_last_device_error().
 *  - Handles own the device memory they allocate at creation and free it in
 *    their destroy call (tgm_state_set_mitigation also allocates the
 *    executor's neighbour-set slots in the mitigator).  Per-batch calls,
 *    tgm_stage_run included, allocate nothing and never synchronise the
 *    device (tgm_alloc_count counts every allocation).  Arrays passed to
 *    tgm_graph_create are BORROWED: they must stay alive and unchanged until
 *    the graph is destroyed.
 *  - A handle must not be used from two threads at once.  Calls on one
 *    handle must be stream-ordered, except that tgm_sample_nodes and
 *    tgm_node_set (which touch only the graph's event arrays and node-set
 *    scratch) may run on another stream beside the state and model calls.
 */
#ifndef TGM_H
#define TGM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Largest number of sample buffer sets tgm_stage_run takes (its nsb). */
#define TGM_MAX_SAMPLE_SETS 16

typedef int32_t tgm_status_t;
#define TGM_OK 0
#define TGM_EINVAL (-1)   /* null pointer, bad size or dimension             */
#define TGM_ERANGE (-2)   /* input content out of range (ids, unsorted time) */
#define TGM_EORDER (-3)   /* iteration protocol violated (see fetch/update)  */
#define TGM_ESIZE (-4)    /* a capacity given at creation is exceeded        */
#define TGM_EDEVICE (-5)  /* a HIP runtime call failed                       */
#define TGM_ENOMEM (-6)   /* device allocation failed at creation            */

typedef struct tgm_graph *tgm_graph_t;
typedef struct tgm_state *tgm_state_t;
typedef struct tgm_model *tgm_model_t;
typedef struct tgm_mitigator *tgm_mitigator_t;

/* Static string for a status code. */
const char *tgm_status_str(tgm_status_t status);
/* First HIP error recorded by a library call since the last query (then
 * cleared), as TGM_EDEVICE, or TGM_OK.  Also polls hipGetLastError(). */
tgm_status_t tgm_last_device_error(void);
/* ABI version: major * 100 + minor. */
int32_t tgm_version(void);
/* *count (host) = the number of device allocations the library has made in
 * this process so far.  Every allocation happens in a create call or in
 * tgm_state_set_mitigation; a caller can read the count before and after any
 * other call to check that it allocated nothing.  TGM_EINVAL if count is
 * NULL. */
tgm_status_t tgm_alloc_count(int64_t *count);

/* ------------------------------------------------------------------------
 * Event graph (Sec. 2: the event set y_uv(t) of a dynamic graph).
 *
 * tgm_graph_create builds, on the device, the temporal adjacency used by the
 * sampler: for every node, the events that touch it (as source or
 * destination; a self-loop once), sorted by (t, e), as 16-byte records
 * (time, event id, other endpoint), with a sparse index of every 64th
 * record's time (8 bytes per 64 records) that the sampler searches first.
 * The handle holds about 32.25 E + 12 N bytes.  src, dst, t and neg are
 * [E] device arrays; efeat is [E x D_e] fp32 on the device, NULL iff D_e == 0.
 * All are borrowed.  The call checks ids in [0, N), t non-decreasing, and
 * synchronises `stream` once (creation is not a per-batch call).
 * Errors: TGM_EINVAL (sizes, null), TGM_ERANGE (content), TGM_ENOMEM.
 */
tgm_status_t tgm_graph_create(int32_t N, int64_t E, const int32_t *src, const int32_t *dst,
                              const double *t, const int32_t *neg, const float *efeat,
                              int32_t D_e, void *stream, tgm_graph_t *out);
tgm_status_t tgm_graph_destroy(tgm_graph_t g);
/* Host outputs; any pointer may be NULL.  n_adj = total adjacency entries. */
tgm_status_t tgm_graph_info(tgm_graph_t g, int32_t *N, int64_t *E, int32_t *D_e,
                            int64_t *n_adj);

/* Roots of the batch of events [first_event, first_event + b): the training
 * samples of an iteration are its events, each with a source, a destination
 * and one negative destination (Sec. 5, training settings: equal numbers of
 * positive and negative pairs; App. E.6: three nodes per sample).
 * Output root[3b] = src[batch] ++ dst[batch] ++ neg[batch], root_ts[3b] = the
 * event time, repeated three times. */
tgm_status_t tgm_batch_roots(tgm_graph_t g, int64_t first_event, int32_t b, int32_t *root,
                             double *root_ts, void *stream);

/* Most-recent-nb temporal neighbour sampling (Sec. 5: the 10 most recent
 * 1-hop neighbours; Appendix D.1: fixed-size most-recent sampler).  For root
 * r = (v, root_ts[r]) the neighbours are the events e' touching v with
 * t[e'] < root_ts[r] (strictly earlier), the nb largest by (t[e'], e'),
 * newest first; the neighbour is the other endpoint (v for a self-loop).
 * Outputs: nbr, eid [R x nb] int32, nts [R x nb] fp64 (event time), cnt [R].
 * Slots j >= cnt[r] hold nbr = eid = -1, nts = 0.  1 <= nb <= 64.  R may be 0. */
tgm_status_t tgm_sample(tgm_graph_t g, const int32_t *root, const double *root_ts, int32_t R,
                        int32_t nb, int32_t *nbr, int32_t *eid, double *nts, int32_t *cnt,
                        void *stream);

/* tgm_batch_roots followed by tgm_sample over the 3b roots, in one pass:
 * same outputs (root, root_ts [3b]; nbr, eid, nts [3b x nb]; cnt [3b]). */
tgm_status_t tgm_sample_batch(tgm_graph_t g, int64_t first_event, int32_t b, int32_t nb,
                              int32_t *root, double *root_ts, int32_t *nbr, int32_t *eid,
                              double *nts, int32_t *cnt, void *stream);

/* Node set of the subgraph (Sec. 2, Eq. 1: emb() of a root reads the memory of
 * the root and of its 1-hop temporal neighbours N(v), so an iteration fetches
 * and updates the memory of every node of the sampled subgraph; App. E.6
 * sizes that subgraph at the roots plus nb neighbours each):
 * U = sorted unique(root[0..R) and every valid nbr).  nodes [cap] receives U, *n_nodes (device int32) its size, root_pos
 * [R] and nbr_pos [R x nb] the position in U of every root and neighbour (-1
 * for empty slots).  cap must be >= min(N, R * (nb + 1)).  Uses the graph's
 * scratch: calls on one graph must be stream-ordered. */
tgm_status_t tgm_node_set(tgm_graph_t g, const int32_t *root, int32_t R, const int32_t *nbr,
                          int32_t nb, int32_t *nodes, int32_t *n_nodes, int32_t cap,
                          int32_t *root_pos, int32_t *nbr_pos, void *stream);

/* The sampling of an iteration's subgraph and its node set (Sec. 3.1: the
 * sample stage of the pipeline, which depends on the event stream only; Sec. 5
 * and App. D.1 for the sampler; Eq. 1 for the node set, as above):
 * tgm_sample_batch followed by tgm_node_set over its outputs, with the node
 * marks made by the sampler itself (one launch fewer): same outputs as the
 * two calls (root, root_ts, nbr, eid, nts, cnt; nodes, *n_nodes, root_pos
 * [3b], nbr_pos [3b x nb]); cap >= min(N, 3b (nb + 1)).  Uses the graph's
 * scratch like tgm_node_set. */
tgm_status_t tgm_sample_nodes(tgm_graph_t g, int64_t first_event, int32_t b, int32_t nb,
                              int32_t *root, double *root_ts, int32_t *nbr, int32_t *eid,
                              double *nts, int32_t *cnt, int32_t *nodes, int32_t *n_nodes,
                              int32_t cap, int32_t *root_pos, int32_t *nbr_pos, void *stream);

/* ------------------------------------------------------------------------
 * Node memory and mailbox (Sec. 2: node memory s_v; Sec. 3.1, Eq. 2: reads
 * of stale memory).  Per node: mem [M] fp32, mem_ts fp64 (time of the last
 * memory update), mail [D_m] fp32 with D_m = 2M + D_e (the pending message),
 * mail_ts fp64 (its event time) and ver int32 (iteration of the last write,
 * -1 = never written; a node has mail iff ver >= 0).  Initially all zero and
 * ver = -1.
 *
 * Staleness s >= 0: a fetch at iteration i sees exactly the writes of
 * iterations <= i-1-s (the paper's staleness k equals s + 1; s = 0 is strictly
 * sequential).  Writes of later iterations are staged in a ring of s + 1
 * write sets and committed, in iteration order, by the fetch that first needs
 * them.  max_batch bounds b of every update.
 */
tgm_status_t tgm_state_create(int32_t N, int32_t M, int32_t D_m, int32_t s, int32_t max_batch,
                              void *stream, tgm_state_t *out);
tgm_status_t tgm_state_destroy(tgm_state_t st);
/* Back to the initial state at iteration 0 (tables zero, ver = -1). */
tgm_status_t tgm_state_reset(tgm_state_t st, void *stream);
/* Commit every staged write set. */
tgm_status_t tgm_state_flush(tgm_state_t st, void *stream);
/* Copy the committed tables out: mem [N x M], mem_ts [N], mail [N x D_m],
 * mail_ts [N], ver [N] (device; any may be NULL). */
tgm_status_t tgm_state_read(tgm_state_t st, float *mem, double *mem_ts, float *mail,
                            double *mail_ts, int32_t *ver, void *stream);
/* Replace the committed tables (same layouts) and restart the protocol at
 * iteration `iter`: staged write sets are dropped, and a fetch at i >= iter
 * sees the loaded tables plus the writes of iterations iter .. i-1-s. */
tgm_status_t tgm_state_load(tgm_state_t st, int64_t iter, const float *mem, const double *mem_ts,
                            const float *mail, const double *mail_ts, const int32_t *ver,
                            void *stream);
/* Checkpoint and resume of the whole versioned state (Alg. 1's state between
 * iterations): the committed tables, the staged write sets that no fetch has
 * needed yet (up to s + 1 of them) and the protocol counters, so that a run
 * resumed from a checkpoint gives bit for bit the results of the run that
 * was not interrupted.  The checkpoint is a HOST buffer of
 * tgm_state_checkpoint_bytes bytes (owned by the caller; a self-describing
 * layout with a magic number and format version).  tgm_state_save orders
 * its copies after the work already on `stream` and returns once they are
 * done; no other stream may be writing the state meanwhile.
 * tgm_state_restore loads a checkpoint into a state created with the same
 * N, M, D_m, s and max_batch (else TGM_EINVAL; a bad magic, format or
 * counters that the protocol cannot reach also give TGM_EINVAL) and returns
 * once the tables are on the device.  A buffer shorter than the checkpoint
 * gives TGM_ESIZE.  The next call continues the protocol where the saved
 * state was: a fetch of last_fetch or later, or the update after the last
 * staged one. */
tgm_status_t tgm_state_checkpoint_bytes(tgm_state_t st, size_t *bytes);
tgm_status_t tgm_state_save(tgm_state_t st, void *buf, size_t bytes, void *stream);
tgm_status_t tgm_state_restore(tgm_state_t st, const void *buf, size_t bytes, void *stream);

/* Memory fetch of iteration `iter` (Alg. 1's fetch_memory, after its wait
 * until the update of iteration iter-k is done, with k = s + 1).  First commits
 * every staged write set of iteration <= iter-1-s, then gathers, for the
 * *n_nodes (device) nodes in nodes[]: mem [cap x M], mem_ts [cap],
 * mail [cap x D_m], mail_ts [cap], ver [cap].  Rows past *n_nodes are not
 * written.  TGM_EORDER if the update of some iteration <= iter-1-s has not
 * been issued, or if iter is below a previously fetched iteration. */
tgm_status_t tgm_fetch_memory(tgm_state_t st, int64_t iter, const int32_t *nodes,
                              const int32_t *n_nodes, int32_t cap, float *mem, double *mem_ts,
                              float *mail, double *mail_ts, int32_t *ver, void *stream);

/* ------------------------------------------------------------------------
 * Model (Eq. 1: msg, mem, emb).  Weights are HOST arrays, copied and packed
 * at creation:
 *   GRU memory updater: W_ih [3M x D_x], W_hh [3M x M], b_ih, b_hh [3M], gate
 *     row blocks in order r, z, n; D_x = D_m + D_t.
 *   Time encoding phi(dt)_d = cos(omega_d dt + beta_d): omega, beta [D_t] fp64.
 *   Attention (d_a = M, H heads of width M / H):
 *     W_q [M x (M + D_t)], b_q [M]; W_k, W_v [M x (M + D_e + D_t)], b_k, b_v [M];
 *     W_o [M x 2M], b_o [M].
 * max_nodes and max_roots bound the node-set size and R of every call.
 * Limits of this implementation: M <= 128 and divisible by H, 1 <= nb <= 64,
 * D_e <= 256, and the attention tile of 80 slots x (D_e + D_t) fp32 must fit
 * the 160 KB of LDS of a workgroup (D_e + D_t <= 384); else TGM_EINVAL.
 */
/* Model families (Sec. 5 trains TGN, JODIE and APAN):
 *   TGM_MODEL_TGN    the GRU updater and the attention embedding above;
 *   TGM_MODEL_JODIE  an RNN updater, mem' = tanh(W_ih x + b_ih + W_hh mem + b_hh)
 *     on the same input x = [mail || phi(mail_ts - mem_ts)], with W_ih
 *     [M x D_x], W_hh [M x M], b_ih, b_hh [M]; the embedding is the time
 *     projection h = s' * (1 + w_t (t - ts')) of tgm_embed_projection, w_t [M]
 *     (JODIE's projection of a node's memory to the query time).  The
 *     attention weights and H are not read (H must still divide M). */
#define TGM_MODEL_TGN 0
#define TGM_MODEL_JODIE 1

typedef struct {
    int32_t M, D_e, D_t, H, nb;
    int32_t max_nodes, max_roots;
    int32_t kind;   /* TGM_MODEL_TGN or TGM_MODEL_JODIE */
} tgm_model_desc;

typedef struct {
    const float *W_ih, *W_hh, *b_ih, *b_hh;
    const double *omega, *beta;
    const float *W_q, *b_q, *W_k, *b_k, *W_v, *b_v, *W_o, *b_o;
    const float *w_t;   /* TGM_MODEL_JODIE: [M] */
} tgm_weights;

tgm_status_t tgm_model_create(const tgm_model_desc *desc, const tgm_weights *w, void *stream,
                              tgm_model_t *out);
tgm_status_t tgm_model_destroy(tgm_model_t m);

/* Memory update of iteration `iter` (Eq. 1 with the stale reads of Eq. 2;
 * Alg. 1's update_mem):
 *  - for every node p < *n_nodes of the fetched set with ver[p] >= 0:
 *      mem_new[p] = GRU([mail[p] || phi(mail_ts[p] - mem_ts[p])], mem[p])
 *        (the RNN cell for TGM_MODEL_JODIE models),
 *      new_mem_ts[p] = mail_ts[p]  (Delta-t as defined under Eq. 1);
 *    otherwise mem_new[p] = mem[p], new_mem_ts[p] = mem_ts[p];
 *  - messages of the b positive events [first_event, first_event + b)
 *    (identity msg: [s'_self || s'_other || efeat[e]], time t[e]) and the
 *    latest-message reduce: per endpoint node the message with the largest
 *    (t, e, role), role src = 0 < dst = 1;
 *  - stages the write set of iteration `iter`: for each endpoint node w,
 *    mem <- mem_new[w], mem_ts <- new_mem_ts[w], mail <- winning message,
 *    mail_ts <- its time, ver <- iter.
 * src_pos / dst_pos [b] are the positions in the node set of each event's
 * source and destination (the first and second thirds of root_pos).
 * Outputs: mem_new [cap x M], new_mem_ts [cap] (may be NULL), winner [cap]
 * int64 (may be NULL): 2e + role of the winning message per node, -1 if none.
 * TGM_EORDER unless iter is the next iteration after the last update (0 after
 * create/reset, `iter` after load) and the fetch of iter has been issued. */
tgm_status_t tgm_update_memory(tgm_state_t st, tgm_model_t m, tgm_graph_t g, int64_t iter,
                               const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                               const float *mem, const double *mem_ts, const float *mail,
                               const double *mail_ts, const int32_t *ver, int64_t first_event,
                               int32_t b, const int32_t *src_pos, const int32_t *dst_pos,
                               float *mem_new, double *new_mem_ts, int64_t *winner,
                               void *stream);

/* Embedding (Eq. 1's emb, "a single layer GAT" in the paper; here one layer of
 * H-head scaled dot-product attention over the sampled neighbours):
 *   q   = W_q [s'_v || phi(0)] + b_q
 *   K_j = W_k [s'_u_j || efeat[eid_j] || phi(root_ts - nts_j)] + b_k, V_j with W_v
 *   a   = concat over heads of softmax_j(q.K_j / sqrt(M/H)) V_j  (0 if cnt = 0)
 *   h   = ReLU(W_o [a || s'_v] + b_o)
 * root_pos [R], root_ts [R], nbr_pos/eid/nts [R x nb], cnt [R] as produced by
 * the calls above; mem_new [cap x M] the updated memory of the node set.
 * Output h [R x M]. */
tgm_status_t tgm_embed(tgm_model_t m, tgm_graph_t g, int32_t R, int32_t nb,
                       const int32_t *root_pos, const double *root_ts, const int32_t *nbr_pos,
                       const int32_t *eid, const double *nts, const int32_t *cnt,
                       const float *mem_new, const int32_t *n_nodes, int32_t cap, float *h,
                       void *stream);

/* JODIE's embedding (TGM_MODEL_JODIE models; TGN models: TGM_EINVAL): the
 * time projection of each root's updated memory to its query time,
 *   h[r] = mem_new[p] * (1 + w_t * (root_ts[r] - new_mem_ts[p])),
 *   p = root_pos[r], formed in fp64 and stored as fp32.
 * root_pos [R] and root_ts [R] as from tgm_sample_nodes; mem_new [cap x M]
 * and new_mem_ts [cap] as from tgm_update_memory.  Output h [R x M].  Errors:
 * TGM_EINVAL (null, dims, model family), TGM_ESIZE (R above max_roots or cap
 * above max_nodes). */
tgm_status_t tgm_embed_projection(tgm_model_t m, int32_t R, const int32_t *root_pos,
                                  const double *root_ts, const float *mem_new,
                                  const double *new_mem_ts, const int32_t *n_nodes, int32_t cap,
                                  float *h, void *stream);

/* ------------------------------------------------------------------------
 * Pipelined executor.  Runs iterations i0 .. i0+n-1 of the stage (the batch of
 * iteration i is events [iB, min(E, (i+1)B))).  The sample and node set of an
 * iteration depend on the event stream only (Sec. 3.1: MSPipe prefetches
 * them), so they run ahead on prefetch_stream in chunks of 1, 2, 4, ... and
 * then nsb/2 iterations (each chunk sampled while the one before it is
 * computed), into sample buffer set (i - i0) % nsb; the fetch, update and embedding of
 * each iteration run in order on `stream` with one set of fetch buffers, in
 * three launches per iteration (the staging of a write set shares a launch
 * with the node projections, and the attention with the next fetch's
 * gather; for JODIE models: the update, the staging, and the projection with
 * the next fetch's gather).  Without mitigation (tgm_state_set_mitigation)
 * and without training (tgm_state_set_training), and when the model's GRU
 * keeps its weights resident (the shapes of the bench workloads) and
 * new_mem_ts is given, every fetch but the last forms only the GRU's time
 * input and the GRU reads the node set's rows from the committed tables in
 * place: until that iteration's staging commits the next write set they hold
 * the very rows a fetch would copy.  After the call the fetch buffers hold
 * the last iteration's fetched rows, in every mode.  The streams synchronise
 * once per chunk.  The prefetch stream starts after everything issued
 * before on `stream`, and
 * `stream` ends after the last embedding.  Results equal those of issuing
 * tgm_sample_nodes, tgm_fetch_memory, tgm_update_memory and tgm_embed (or
 * tgm_embed_projection) per iteration in order on one stream.
 * 2 <= nsb <= TGM_MAX_SAMPLE_SETS and even (TGM_EINVAL if odd or below 2,
 * TGM_ESIZE if above); nb, cap as for the calls above; mem_new [cap x M],
 * new_mem_ts [cap] (may be NULL), winner [cap] (may be NULL) and h [3B x M]
 * hold the last iteration's outputs.  Optional per-iteration copies (NULL:
 * none): h_trace [n x 3B x M] receives every iteration's embeddings (rows
 * past 3b of a partial last batch untouched), s_trace [n x cap x M] every
 * iteration's new memories mem_new (rows past its node-set size untouched).
 * The two streams must differ.  The call allocates nothing and does not
 * synchronise the host with the device.  Errors of the underlying calls are
 * returned as they occur (the iterations before stay enqueued). */
typedef struct {
    int32_t *root;      /* [3B] */
    double *root_ts;    /* [3B] */
    int32_t *nbr, *eid; /* [3B x nb] */
    double *nts;        /* [3B x nb] */
    int32_t *cnt;       /* [3B] */
    int32_t *nodes;     /* [cap] */
    int32_t *n_nodes;   /* [1] */
    int32_t *root_pos;  /* [3B] */
    int32_t *nbr_pos;   /* [3B x nb] */
} tgm_sample_buffers;

typedef struct {
    float *mem;         /* [cap x M] */
    double *mem_ts;     /* [cap] */
    float *mail;        /* [cap x D_m] */
    double *mail_ts;    /* [cap] */
    int32_t *ver;       /* [cap] */
} tgm_fetch_buffers;

tgm_status_t tgm_stage_run(tgm_graph_t g, tgm_state_t st, tgm_model_t m, int64_t i0, int64_t n,
                           int32_t B, int32_t nb, int32_t cap, const tgm_sample_buffers *sb,
                           int32_t nsb, const tgm_fetch_buffers *fb, float *mem_new,
                           double *new_mem_ts, int64_t *winner, float *h, float *h_trace,
                           float *s_trace, void *stream, void *prefetch_stream);

/* ------------------------------------------------------------------------
 * Training step (the step that follows the stage in MTGNN training: Sec. 5,
 * training settings, link prediction on equal numbers of positive and
 * negative pairs, learning rate 1e-4; App. C.2, the embedding, the loss and
 * the backward step).  TGN models only.
 *
 * The iteration's training samples are its b positive pairs (src_e, dst_e)
 * and b negative pairs (src_e, neg_e), i.e. roots e, b + e and 2b + e.  The
 * link predictor scores a pair from the two embeddings,
 *   z = W_src h_u + W_dst h_v + b_p,  score(u, v) = w_out . ReLU(z) + b_out,
 * and the loss is L = (1/b) sum_e [softplus(-score(src_e, dst_e)) +
 * softplus(score(src_e, neg_e))] (binary cross-entropy on the scores).  The
 * gradient of L reaches every weight of the attention (through h), of the
 * memory updater (through the new memories s' of the nodes that hold mail)
 * and of the predictor; the fetched memories and mails are inputs of the
 * iteration, and omega and beta are not trained.  Then one optimizer step
 * (SGD: theta -= lr g; Adam: the bias-corrected moments of Kingma and Ba) and
 * the model's packed operands are rebuilt from the new weights, so the next
 * iteration runs with them.
 *
 * Parameter vector (float, in this order): W_ih [3M x D_x], W_hh [3M x M],
 * b_ih [3M], b_hh [3M], W_q [M x (M + D_t)], b_q [M], W_k [M x D_kv], b_k [M],
 * W_v [M x D_kv], b_v [M], W_o [M x 2M], b_o [M], W_src [M x M],
 * W_dst [M x M], b_p [M], w_out [M], b_out [1], with D_kv = M + D_e + D_t.
 * Every reduction has a fixed order: results are bit-reproducible.
 */
typedef struct tgm_trainer *tgm_trainer_t;
#define TGM_OPT_SGD 0
#define TGM_OPT_ADAM 1
#define TGM_N_PARAM_TENSORS 17

typedef struct {
    const float *W_src, *W_dst; /* host [M x M] */
    const float *b_p, *w_out;   /* host [M] */
    float b_out;
} tgm_predictor;

typedef struct {
    int32_t kind;                 /* TGM_OPT_SGD or TGM_OPT_ADAM */
    float lr, beta1, beta2, eps;  /* beta1, beta2, eps: Adam only */
} tgm_optimizer;

/* A trainer for model m (a TGN model, M <= 128), with the model's weights w
 * (HOST arrays, the ones given to tgm_model_create) and the predictor's p
 * copied into its device parameter vector; it owns the gradient, the
 * optimizer's moments and the work space for batches of up to
 * max_roots / 3 events and node sets of up to max_nodes rows (m's limits).
 * The trainer rewrites m's operands after every step: m must not be used by
 * another trainer.  Errors: TGM_EINVAL (null, JODIE model, parameters),
 * TGM_ENOMEM, TGM_EDEVICE. */
tgm_status_t tgm_trainer_create(tgm_model_t m, const tgm_weights *w, const tgm_predictor *p,
                                const tgm_optimizer *opt, void *stream, tgm_trainer_t *out);
tgm_status_t tgm_trainer_destroy(tgm_trainer_t tr);
/* Host outputs (each may be NULL): the parameter count, the sizes of the
 * TGM_N_PARAM_TENSORS tensors in vector order, the optimizer steps taken. */
tgm_status_t tgm_trainer_info(tgm_trainer_t tr, int64_t *n_params, int64_t *sizes,
                              int64_t *steps);
/* Device copies (each may be NULL, ordered on `stream`): the parameter vector
 * [n_params], the gradient of the last step [n_params], its loss [1]. */
tgm_status_t tgm_trainer_read(tgm_trainer_t tr, float *params, float *grad, float *loss,
                              void *stream);
/* The training step of the iteration whose sample buffers sb (root_pos,
 * root_ts, nbr_pos, eid, nts, cnt, n_nodes as from tgm_sample_nodes), fetch
 * buffers fb (the rows as fetched, after the mitigation when it is on), new
 * memories mem_new [cap x M] (tgm_update_memory) and embeddings h [3b x M]
 * (tgm_embed) are given; b events; loss (device [1], may be NULL) receives
 * the loss.  Stream-ordered; allocates nothing.  Errors: TGM_EINVAL,
 * TGM_ESIZE (3b above max_roots or cap above max_nodes). */
tgm_status_t tgm_train_step(tgm_trainer_t tr, tgm_model_t m, tgm_graph_t g, int32_t b,
                            const tgm_sample_buffers *sb, const tgm_fetch_buffers *fb,
                            const float *mem_new, const float *h, int32_t cap, float *loss,
                            void *stream);
/* Makes tgm_stage_run take the training step after every iteration (tr NULL:
 * off, the default).  With loss_log (device, may be NULL) the loss of
 * iteration i goes to loss_log[i % log_len].  In training mode the executor
 * launches each next fetch after the training step (the step reads the
 * iteration's fetch buffers), instead of in the attention launch. */
tgm_status_t tgm_state_set_training(tgm_state_t st, tgm_trainer_t tr, float *loss_log,
                                    int64_t log_len);

/* ------------------------------------------------------------------------
 * APAN (Sec. 5 trains APAN; App. B: an RNN memory updater with an attention
 * mechanism and asynchronous propagation).  A handle with its own state:
 *   mailbox   per node the K_mb latest mails (the identity message
 *             [s'_self || s'_other || efeat[e]] with its event time), oldest
 *             first; a full mailbox drops its oldest;
 *   propagation  the mail an event generates for its endpoint v goes to v
 *             and (propagate != 0) to v's sampled neighbours at the event's
 *             time (the nb most recent, as tgm_sample_nodes returns them for
 *             root v), in (t, e, role, slot) order;
 *   updater   for a node with mail: q = W_q [s || phi(0)] + b_q,
 *             K_j = W_k [mail_j || phi(t_newest - t_j)] + b_k,
 *             a = sum_j softmax_j(q . K_j / sqrt(M)) mail_j,
 *             s' = GRU([a || phi(t_newest - mem_ts)], s), new_mem_ts = t_newest
 *             (W_ih [3M x D_x], W_hh [3M x M], gates r, z, n as for TGN);
 *             a node without mail keeps s;
 *   embedding h = s' of each root;
 *   write set of iteration i: the new memory of the batch's endpoints
 *             (version i) and the iteration's mail deliveries, committed
 *             before the fetch of iteration i + s + 1 (Eq. 2).
 * Weights: W_ih, W_hh, b_ih, b_hh, W_q [M x (M + D_t)], b_q [M],
 * W_k [M x (2M + D_e + D_t)], b_k [M], omega, beta of tgm_weights (HOST,
 * copied); the other fields are not read.  Limits: M <= 128, D_e <= 256,
 * 1 <= nb <= 64, 1 <= K_mb <= 16.
 */
typedef struct tgm_apan *tgm_apan_t;
typedef struct {
    int32_t N, M, D_e, D_t, nb;
    int32_t K_mb, propagate;
    int32_t s, max_batch, max_nodes;   /* staleness; events per batch; node-set rows */
} tgm_apan_desc;
tgm_status_t tgm_apan_create(const tgm_apan_desc *desc, const tgm_weights *w, void *stream,
                             tgm_apan_t *out);
tgm_status_t tgm_apan_destroy(tgm_apan_t a);
/* Iteration `iter` (the batch [iter B, min(E, (iter + 1) B)), B = max_batch)
 * from its sample and node set sb (tgm_sample_nodes of that batch with the
 * same nb): commits the due write sets, fetches the node set's memories and
 * mailboxes, updates them, writes mem_new [cap x M], new_mem_ts [cap] (may
 * be NULL) and h [3b x M], and stages the write set.  Iterations are issued
 * consecutively from 0 (else TGM_EORDER).  Errors: TGM_EINVAL, TGM_ESIZE
 * (cap above max_nodes), TGM_ERANGE (iter past the stream). */
tgm_status_t tgm_apan_step(tgm_apan_t a, tgm_graph_t g, int64_t iter,
                           const tgm_sample_buffers *sb, int32_t cap, float *mem_new,
                           double *new_mem_ts, float *h, void *stream);
/* Commit every staged write set. */
tgm_status_t tgm_apan_flush(tgm_apan_t a, void *stream);
/* The committed tables (device, each may be NULL; mb and mb_ts together):
 * mem [N x M], mem_ts [N], ver [N], mb [N x K_mb x D_m] and mb_ts
 * [N x K_mb] oldest mail first (zero past the count), mb_cnt [N]. */
tgm_status_t tgm_apan_read(tgm_apan_t a, float *mem, double *mem_ts, int32_t *ver, float *mb,
                           double *mb_ts, int32_t *mb_cnt, void *stream);
/* The initial state again (zero memories, versions -1, empty mailboxes);
 * staged write sets are dropped and the next step is iteration 0. */
tgm_status_t tgm_apan_reset(tgm_apan_t a, void *stream);
/* Replace the committed tables (device, the layouts of tgm_apan_read; none
 * may be NULL; counts outside [0, K_mb] are clamped, mails past a count are
 * ignored) and restart the protocol at iteration `iter`: staged write sets
 * are dropped, and the fetch of a step i >= iter sees the loaded tables plus
 * the write sets of iterations iter .. i-1-s (Eq. 2).  The next step is
 * iteration `iter`.  The copies are ordered on `stream`. */
tgm_status_t tgm_apan_load(tgm_apan_t a, int64_t iter, const float *mem, const double *mem_ts,
                           const int32_t *ver, const float *mb, const double *mb_ts,
                           const int32_t *mb_cnt, void *stream);
/* The last step's fetched rows (device, each may be NULL), in node-set order:
 * mem [max_nodes x M], mem_ts, ver [max_nodes], mb [max_nodes x K_mb x D_m],
 * mb_ts [max_nodes x K_mb] (oldest first), mb_cnt [max_nodes]. */
tgm_status_t tgm_apan_fetched(tgm_apan_t a, float *mem, double *mem_ts, int32_t *ver, float *mb,
                              double *mb_ts, int32_t *mb_cnt, void *stream);

/* ------------------------------------------------------------------------
 * Similarity-based staleness mitigation (MSPipe-S, Sec. 3.3), applied to the
 * fetched memories of a batch between tgm_fetch_memory and
 * tgm_update_memory.  For the fetched node set (positions p < *n_nodes):
 *   gap      dt_p = T - mem_ts[p], T = the time of event first_event (the
 *            batch's first event), formed in fp64;
 *   gamma    the nearest-rank p-quantile of the gaps: the ceil(p n)-th
 *            smallest, with the rank formed as ceil(p * n) in fp64;
 *   stale    dt > gamma; active: dt < gamma;
 *   N(u)     the distinct other endpoints of u's nb most recent events
 *            strictly before T;
 *   Omega(v) the K active nodes sharing the most neighbours with v (at least
 *            one), ties to the larger mem_ts, then the smaller node id;
 *   mem[v] = lambda mem[v] + (1 - lambda) mean_{u in Omega(v)} mem[u] for
 *            every stale v with Omega(v) non-empty (fp32, the sum in Omega's
 *            order); other rows are untouched.
 * The mitigator owns its work space: the neighbour sets, gamma, the stale
 * positions and Omega of the last call.  Calls on one mitigator must be
 * stream-ordered.  Under tgm_stage_run the neighbour sets of each iteration
 * are built on the prefetch stream beside its sample, in one of the
 * TGM_MAX_SAMPLE_SETS slots that tgm_state_set_mitigation makes; the
 * threshold and the blend run on the main stream.
 */
/* max_nodes >= any cap passed later, at most 1 << 20; 1 <= nb <= 64 (the
 * neighbour sets' nb); 1 <= K <= 16.  Errors: TGM_EINVAL, TGM_ENOMEM,
 * TGM_EDEVICE. */
tgm_status_t tgm_mitigator_create(int32_t max_nodes, int32_t nb, int32_t K,
                                  tgm_mitigator_t *out);
tgm_status_t tgm_mitigator_destroy(tgm_mitigator_t mt);
/* nodes [cap] and n_nodes [1] as from tgm_sample_nodes; mem [cap x M] (updated
 * in place) and mem_ts [cap] as from tgm_fetch_memory; 0 <= p <= 1,
 * 0 <= lambda <= 1.  Errors: TGM_EINVAL (null, dims, parameters), TGM_ERANGE
 * (first_event outside the graph), TGM_ESIZE (cap above max_nodes). */
tgm_status_t tgm_mitigate(tgm_mitigator_t mt, tgm_graph_t g, int64_t first_event,
                          const int32_t *nodes, const int32_t *n_nodes, int32_t cap,
                          float *mem, const double *mem_ts, int32_t M, double p, float lambda,
                          void *stream);
/* The mitigation of tgm_mitigate without a mitigator handle, for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc.  Same computation and results as
 * tgm_mitigate with a mitigator of the same nb and K.  Its work space (the
 * neighbour sets, gamma, the stale list, Omega, the chunk lists and counters)
 * lives in a fixed array of TGM_MITIGATE_NOALLOC_BYTES bytes that the library
 * holds on every GPU it runs on until the process ends; the call allocates
 * nothing.  The first call on a device looks that device's array up (the
 * calling thread's current device must be the stream's device).  All calls on
 * one GPU share the array and it keeps the last call's contents: calls that
 * overlap on one GPU (other streams, other threads) race; calls ordered on
 * one stream do not.  Each call clears what it needs at zero itself.  Limits:
 * cap <= TGM_MITIGATE_NOALLOC_MAX_NODES (else TGM_ESIZE); 1 <= nb <= 64 and
 * 1 <= K <= 16 (else TGM_EINVAL).  Other arguments and errors as for
 * tgm_mitigate. */
#define TGM_MITIGATE_NOALLOC_MAX_NODES 32768
#define TGM_MITIGATE_NOALLOC_BYTES (12u << 20)
tgm_status_t tgm_mitigate_noalloc(tgm_graph_t g, int64_t first_event, const int32_t *nodes,
                                  const int32_t *n_nodes, int32_t cap, float *mem,
                                  const double *mem_ts, int32_t M, int32_t nb, int32_t K,
                                  double p, float lambda, void *stream);
/* Device copies of the last call's results (each pointer may be NULL): gamma
 * [1], n_stale [1], stale [max_nodes] (positions, ascending; the first
 * *n_stale are valid), omega [max_nodes x K] (positions, -1 padded; row q
 * belongs to stale[q]). */
tgm_status_t tgm_mitigator_read(tgm_mitigator_t mt, double *gamma, int32_t *n_stale,
                                int32_t *stale, int32_t *omega, void *stream);
/* Makes tgm_stage_run mitigate every fetch with mt, p and lambda (mt NULL:
 * off, the default).  mt must stay alive while st uses it.  A set-up call:
 * the first call with a mitigator allocates its executor slots (one
 * neighbour-set table per sample buffer set) after synchronising the device.
 * Errors: TGM_EINVAL, TGM_ENOMEM, TGM_EDEVICE. */
tgm_status_t tgm_state_set_mitigation(tgm_state_t st, tgm_mitigator_t mt, double p,
                                      float lambda);

/* ------------------------------------------------------------------------
 * Minimal-staleness bound (Sec. 3.2, Eq. 3 and Eq. 4, constraints C1-C3).
 * Host code; touches no device.
 *
 * tau [5]: the durations of the stages 1 sample, 2 feature fetch, 3 memory
 * fetch, 4 compute, 5 memory update (any time unit, each >= 0).  For
 * iterations i = 1..n the start times b_i^(j) and end times
 * e_i^(j) = b_i^(j) + tau^(j) follow Eq. 3: b_i^(1) = e_{i-1}^(1);
 * b_i^(2) = max(e_i^(1), e_{i-1}^(3)); b_i^(j) = max(e_i^(j-1), e_{i-1}^(j))
 * for j = 3..5; every stage of "iteration 0" ends at 0.  Then k_i is the
 * smallest k with 1 <= k < min(i, k_max) such that the memory fetch, started
 * once the update of iteration i - k is done (C1: at
 * max(b_i^(3), e_{i-k}^(5))), ends by b_i^(4) (C2:
 * e_{i-k}^(5) <= b_i^(4) - tau^(3)).  An empty range (i <= 1 or k_max <= 1)
 * is a warm-up iteration: k_i = 0, no wait.  If no k in the range meets C2,
 * k_i = min(i, k_max) - 1 and the fetch stalls the compute stage.
 *
 * Outputs (host arrays, iteration i at index i - 1): k [n]; fetch_start [n],
 * stall [n] (the compute stage's delay, 0 when stall-free), b [n x 5] and
 * e [n x 5] (stage j at column j - 1) may be NULL.  Errors: TGM_EINVAL (null
 * tau or k, n < 0, k_max < 1, a negative or NaN duration).
 */
tgm_status_t tgm_min_staleness(const double *tau, int64_t n, int32_t k_max, int32_t *k,
                               double *fetch_start, double *stall, double *b, double *e);

/* ------------------------------------------------------------------------
 * Per-kernel timing.  When enabled, every kernel the library launches is
 * bracketed by two HIP events recorded on its own stream; tgm_profile_get
 * synchronises those events and reports, per kernel name, the number of
 * launches and their summed duration.  Off by default; enabling it adds two
 * event records per launch.  Not thread-safe.
 */
tgm_status_t tgm_profile_enable(int32_t on);
/* Drops everything recorded so far. */
tgm_status_t tgm_profile_reset(void);
/* Folds pending records into the totals; returns the number of kernel names. */
int32_t tgm_profile_count(void);
/* Totals of the k-th kernel name (0 <= k < tgm_profile_count()).  *name is a
 * static string. */
tgm_status_t tgm_profile_get(int32_t k, const char **name, int64_t *launches, double *total_ms);

#ifdef __cplusplus
}
#endif
#endif /* TGM_H */
