/*
 * ef_attention.h - C ABI of the MI355X (gfx950) fused attention library.
 *
 * The library computes the fused attention program of EquiForge (arXiv
 * 2609.12330): for every batch b and query head hq, with kv head
 * hk = hq / (Hq / Hkv) (replication by index, section 3.1 "Replicate"),
 *
 *     s_ij = scale * <q_i, k_j>,   O_i = sum_j exp(s_ij - m_i) v_j / sum_j exp(s_ij - m_i),
 *     m_i  = max_j s_ij,
 *
 * which is form M0 of figure "attention-rewrites" (section 3). The kernels
 * evaluate it as form M2 of the same figure: the key axis is cut into tiles
 * and a rolling (max, sum, value) reducer is carried over them (section 4.2,
 * repair fusion with h(c, s, s') = c * exp(s - s')). The split-KV entry point
 * additionally stores one reduced state per key partition and combines them
 * in a second kernel (section 3.3 "Collection"; section 4.4 storage rule).
 *
 * Conventions shared by every entry point
 *   - Tensors are dense and row-major with the head dimension innermost:
 *       q  [B][Hq ][Sq ][D] bf16      k, v [B][Hkv][Skv][D] bf16
 *       o  [B][Hq ][Sq ][D] fp32
 *     bf16 is the IEEE binary32 upper half (1-8-7). All pointers are DEVICE
 *     pointers, 16-byte aligned; the caller owns every buffer and keeps it
 *     alive until the stream has passed the call. The library allocates
 *     nothing and keeps no state between calls (apart from the static scratch
 *     of ef_attention_splitkv_noalloc); calls are thread-safe.
 *   - D must be 64 or 128. Hq and Hkv must be >= 1 with Hq % Hkv == 0.
 *     B, Sq and Skv may be 0: with B*Hq*Sq == 0 nothing is written, with
 *     Skv == 0 every output row is 0. Per head, S*D must stay below 2^31.
 *   - causal != 0 applies a bottom-right aligned mask: key j is visible to
 *     query i iff j <= i + (Skv - Sq). A query row that sees no key gets 0.
 *   - scale multiplies the fp32-accumulated q.k products; it must be finite
 *     (0 gives every visible key the same weight). The scaled scores are fp32
 *     values: |scale * q.k| beyond the fp32 range is outside the contract.
 *   - Every call validates its arguments on the host, synchronously, before
 *     anything is enqueued. On an error nothing is launched and no buffer is
 *     written. After validation the work is enqueued on `stream` (a
 *     hipStream_t; NULL is the default stream) and the call returns without
 *     waiting; a launch failure reported by HIP returns EF_ERR_HIP.
 *   - Results are deterministic: the same inputs give bitwise equal outputs.
 *   - Local attention (the *_local entry points; the sliding-window GQA and
 *     attention-sink layers of section 7.3) is causal attention restricted
 *     to a window of `window` keys plus `sinks` sink keys: with
 *     n_i = i + (Skv - Sq), key j is visible to query i iff j <= n_i and
 *     (j > n_i - window or j < sinks). window >= 1, sinks >= 0; a window of
 *     Skv keys or more is plain causal attention. Keys that no query row of
 *     a workgroup can see are not read: the kernels visit the sink keys and
 *     the window and skip the masked middle.
 */
#ifndef EF_ATTENTION_H
#define EF_ATTENTION_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

#define EF_ABI_VERSION 2

typedef enum {
  EF_OK = 0,
  EF_ERR_NULL_POINTER = 1,         /* a required pointer is NULL */
  EF_ERR_INVALID_SHAPE = 2,        /* a negative size, Hq or Hkv < 1, or a head too large */
  EF_ERR_GQA_RATIO = 3,            /* Hq is not a multiple of Hkv */
  EF_ERR_UNSUPPORTED_HEAD_DIM = 4, /* D is not 64 or 128 */
  EF_ERR_MISALIGNED = 5,           /* a pointer is not 16-byte aligned */
  EF_ERR_INVALID_PARTITION = 6,    /* partition_size is not 0 or a positive multiple of 64, or
                                      it gives more than 65535 partitions */
  EF_ERR_WORKSPACE_TOO_SMALL = 7,  /* workspace is NULL or smaller than required */
  EF_ERR_INVALID_SCALE = 8,        /* scale is NaN or infinite */
  EF_ERR_HIP = 9,                  /* HIP reported an error when the work was enqueued */
  EF_ERR_INVALID_MASK = 10,        /* local attention: window < 1 or sinks < 0 */
  EF_ERR_INVALID_DIFF = 11,        /* differential attention: lambda_init or eps not finite, or eps < 0 */
  EF_ERR_INVALID_SPLIT = 12,       /* d_splits not 1, 2 or 4, or more than 8 query rows per kv head */
  EF_ERR_SCRATCH_TOO_SMALL = 13    /* the problem needs more than EF_STATIC_SCRATCH_BYTES of scratch */
} ef_status;

/* Version of this ABI (EF_ABI_VERSION). */
int ef_abi_version(void);

/* Static, NUL-terminated description of a status code; never NULL. */
const char* ef_status_string(int status);

/*
 * Single-pass attention: form M2 of figure "attention-rewrites". The query
 * rows that share a kv head are tiled along the query axis (grid axis m), each
 * workgroup carries the rolling reducer over all key tiles it can see and
 * writes O = value / sum once at the end (section 6.1: output-tile axes map
 * to the grid, reduction axes to an in-workgroup loop).
 *   q, k, v, o : device buffers in the layouts above.
 *   B, Hq, Hkv, Sq, Skv, D, scale, causal : as above.
 *   stream     : hipStream_t or NULL.
 */
ef_status ef_attention_fwd(const void* q, const void* k, const void* v, float* o,
                           int B, int Hq, int Hkv, int Sq, int Skv, int D,
                           float scale, int causal, void* stream);

/*
 * ef_attention_fwd with local attention (causal mask, sliding window of
 * `window` keys, `sinks` sink keys; see the conventions above). Each
 * workgroup reads the key tiles of the sink run and of its rows' windows
 * only; both runs feed one rolling reducer, so sink and window keys share one
 * softmax normalisation (section 7.3, attention sinks).
 * Returns EF_ERR_INVALID_MASK when window < 1 or sinks < 0.
 */
ef_status ef_attention_fwd_local(const void* q, const void* k, const void* v, float* o,
                                 int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                 float scale, int window, int sinks, void* stream);

/*
 * Partition size, in keys, that ef_attention_splitkv uses for these sizes:
 * `partition_size` itself when it is positive, else the library's choice
 * (the candidate ef_attention_splitkv_modeled_us rates fastest).
 * Returns 0 when the arguments are invalid.
 */
int ef_attention_splitkv_partition_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                        int partition_size);

/*
 * Bytes of workspace ef_attention_splitkv needs for these sizes (0 when the
 * arguments are invalid or nothing is computed). With rows = B*Hq*Sq,
 * P = ceil(Skv / T) and T the resolved partition size, the workspace holds
 *     counters [512][64] uint32 at byte 0 (EF_COUNTER_REGION_BYTES)
 *     m   [rows][P]    fp32 at byte  C = EF_COUNTER_REGION_BYTES
 *     l   [rows][P]    fp32 at byte  C + A, A = round_up(rows*P*4, 256)
 *     acc [rows][P][D] fp32 at byte  C + 2*A
 * with row = (b*Hq + hq)*Sq + sq: a reference point m for the scaled scores
 * s of the row's visible keys in partition p (natural-log units; at most the
 * partition maximum and within 8*ln(2) of it), l = sum exp(s - m) and
 * acc = sum exp(s - m) * v. (m, l, acc) and (m', l*e^(m-m'), acc*e^(m-m'))
 * describe the same state. A partition with no visible key holds the reducer
 * identity (-inf, 0, 0). The counters are arrival counters of the fused
 * combine (see ef_attention_splitkv): word 0 of each 256-byte slot
 * counters[b*Hkv + hk] serves one (batch, kv head); the rest is padding. The
 * counter region has the same place and size for every problem, and no
 * partial state is ever stored in it.
 */
#define EF_COUNTER_REGION_BYTES ((size_t)512 * 256)

size_t ef_attention_splitkv_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                           int partition_size);

/*
 * Split-KV attention for decode-shaped problems (few query rows per kv head,
 * long key axis). The key axis is cut into P partitions of T keys; one
 * workgroup per (partition, kv head, batch) reads its K/V slice once, serves
 * all Hq/Hkv * Sq query rows of that kv head, and stores the reduced state
 * (m, l, acc) of every row in the workspace (the Collection of section 3.3
 * and the storage rule of section 4.4). A second kernel combines the P states
 * of each row with the same reducer and writes o (section 4.1, reduction
 * refinement along K; section 4.2, repair fusion).
 *   partition_size   : T in keys; 0 lets the library choose; otherwise a
 *                      positive multiple of 64.
 *   workspace        : device buffer of at least
 *                      ef_attention_splitkv_workspace_size(...) bytes,
 *                      16-byte aligned; on return (stream-ordered) it holds
 *                      the partial states in the layout documented there.
 *                      Its counter region (the first EF_COUNTER_REGION_BYTES)
 *                      must be zero before the first call that uses it
 *                      (zero-fill the new buffer once); every completed call
 *                      leaves it zero again, so a workspace serves any number
 *                      of calls of any shapes whose workspace fits in it, in
 *                      stream order. Calls that overlap in time must not share
 *                      a workspace.
 *   workspace_bytes  : its size in bytes.
 * When G*Sq <= 4, P <= 64 and B*Hkv <= 512 the combine runs inside the
 * producer: the last workgroup of each (batch, kv head) to store its state,
 * found with the group's arrival counter, combines that group's rows and
 * resets the counter (one kernel instead of two). Otherwise a separate combine
 * kernel follows. A counter that is not zero when the call begins (a counter
 * region never cleared) cannot tell which workgroup is last; the producer
 * then fills that group's output rows with NaN rather than combine states
 * that may be stale.
 * Other arguments as for ef_attention_fwd.
 */
ef_status ef_attention_splitkv(const void* q, const void* k, const void* v, float* o,
                               int B, int Hq, int Hkv, int Sq, int Skv, int D,
                               float scale, int causal, int partition_size,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * Split-KV attention with local attention (causal mask, window, sinks; see
 * the conventions above). The keys any query row of a (batch, kv head) can
 * see lie in two runs: the sink run [0, La), La = min(round_up(sinks, 64),
 * Skv), and the window run [Bs, Skv), Bs = max(La, round_down(max(0,
 * Skv - Sq - window + 1), 64)). The partitions of T keys cut the
 * concatenation of the two runs, Lv = La + Skv - Bs keys, so P = ceil(Lv / T)
 * and no workgroup is spent on the masked middle. Workspace layout, counters
 * and the fused-combine rule are those of ef_attention_splitkv with this P
 * (partition p covers concatenated keys [p*T, p*T + T)).
 * Returns EF_ERR_INVALID_MASK when window < 1 or sinks < 0.
 */
ef_status ef_attention_splitkv_local(const void* q, const void* k, const void* v, float* o,
                                     int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                     float scale, int window, int sinks, int partition_size,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * Partition size and workspace bytes of ef_attention_splitkv_local, as for
 * the causal entry points but over the Lv keys of the two visible runs.
 * Return 0 when the arguments are invalid (including window < 1 or sinks < 0).
 */
int ef_attention_splitkv_local_partition_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                              int window, int sinks, int partition_size);
size_t ef_attention_splitkv_local_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv,
                                                 int D, int window, int sinks,
                                                 int partition_size);

/*
 * The producer step of ef_attention_splitkv alone: the same validation and
 * the same kernels, writing only the partial states into the workspace
 * (layout of ef_attention_splitkv_workspace_size). Combining them with
 * ef_attention_combine gives ef_attention_splitkv's output; partial states of
 * disjoint key ranges (e.g. computed on different devices, each over its own
 * slice of the key axis) may be concatenated along P before the combine,
 * since the combine applies the same reducer to any set of stored states.
 */
ef_status ef_attention_splitkv_partials(const void* q, const void* k, const void* v,
                                        int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                        float scale, int causal, int partition_size,
                                        void* workspace, size_t workspace_bytes, void* stream);

/*
 * The combine step alone, over caller-provided fp32 partial states:
 *   m [rows][P], l [rows][P], acc [rows][P][D] (device, 16-byte aligned),
 *   o [rows][D] fp32 output.
 * For each row: M = max_p m_p, w_p = exp(m_p - M) (0 where m_p = -inf),
 * o = (sum_p w_p acc_p) / (sum_p w_p l_p), and o = 0 when M = -inf
 * (section 4.2, the fused reducer applied to stored states).
 * rows >= 0, P >= 1, D in {64, 128}.
 */
ef_status ef_attention_combine(const float* m, const float* l, const float* acc, float* o,
                               int rows, int num_partitions, int D, void* stream);

/*
 * Modelled duration in microseconds of one split-KV call with
 * `partition_size` keys per partition (window = sinks = 0 for the causal or
 * full entry point; a local window otherwise). The model is the roofline rule
 * of section 6.2, static family ranking (over legal schedules, minimise the
 * largest work/throughput ratio over resources): the larger of the HBM time
 * (K/V, q, o and the partial states written and read) and one workgroup's
 * streaming time times the rounds of workgroups the chip holds, plus the
 * combine, with rates measured on MI355X. With partition_size = 0 the
 * split-KV entry points take the candidate (64, 128, 256, 512, ... keys, and
 * one partition holding every key) this model rates fastest.
 * Returns a negative value for invalid arguments.
 */
double ef_attention_splitkv_modeled_us(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                       int window, int sinks, int partition_size);

/*
 * Query rows per workgroup of the matrix-core kernel for these sizes, as the
 * entry points choose them (64 or 128; the Hq/Hkv query heads of a kv head
 * are packed into its rows). The choice follows the roofline rule of section
 * 6.2 over the legal values: each is charged the larger of its matrix work
 * (rows padded to whole workgroups) over the bf16 peak and its global-memory
 * traffic (the K/V that every row tile stages, plus q and o) over the HBM
 * peak; the smallest wins, and with equal times the one with less matrix
 * work. `keys`: the keys a row tile streams (Skv for a full or causal
 * prefill, the partition size in a split-KV call). Returns 0 for invalid
 * sizes or keys < 0.
 */
int ef_attention_rows_per_workgroup(int B, int Hq, int Hkv, int Sq, int Skv, int D, int keys);

/*
 * Measures the best partition size for these inputs on this device: the six
 * candidates the model rates fastest (among those whose workspace fits in
 * workspace_bytes) are timed by successive halving (section 6.3: every
 * remaining candidate runs, the faster half stays, the repetitions double)
 * and the winner is written to *partition_size. window = 0 selects the
 * full/causal path (causal as given; sinks must be 0), window > 0 the local
 * path. Runs the split-KV call many times on `stream` (o and the workspace
 * are overwritten), waits for it with HIP events, and so cannot be captured
 * in a graph. Errors as for the split-KV entry points; EF_ERR_NULL_POINTER
 * when partition_size is NULL.
 */
ef_status ef_attention_splitkv_tune(const void* q, const void* k, const void* v, float* o,
                                    int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                    float scale, int causal, int window, int sinks,
                                    void* workspace, size_t workspace_bytes, void* stream,
                                    int* partition_size);

/*
 * Differential attention (section 7.3, the differential attention layer of
 * the cited differential transformer): two attention branches over one value
 * tensor,
 *   A1 = attention(q1, k1, v),  A2 = attention(q2, k2, v)
 * (same scale, causal flag and grouped-query mapping as ef_attention_fwd),
 * mixed with the learned weight
 *   lambda = exp(<lambda_q1, lambda_k1>) - exp(<lambda_q2, lambda_k2>) + lambda_init
 * and normalised per head and query row over the head dimension:
 *   y = A1 - lambda * A2
 *   o = (1 - lambda_init) * norm_weight * y / sqrt(mean(y^2) + eps),
 * and o = 0 for a row where mean(y^2) + eps is 0 (y = 0 with eps = 0). The
 * weight, the difference and the normalisation are applied by one kernel as
 * the first branch's output is formed, so no A1 tensor is written.
 *   q1, q2 : [B][Hq][Sq][D] bf16; k1, k2, v : [B][Hkv][Skv][D] bf16;
 *   o      : [B][Hq][Sq][D] fp32, also used to hold A2 between the branches.
 *   lambda_q1, lambda_k1, lambda_q2, lambda_k2, norm_weight : [D] fp32 device
 *            buffers, shared by all heads; norm_weight 16-byte aligned.
 *   lambda_init, eps : finite, eps >= 0 (else EF_ERR_INVALID_DIFF).
 *   partition_size : 0 (model choice, as for ef_attention_splitkv) or a
 *            positive multiple of 64. When the resolved partition covers every
 *            key each branch is one single-pass launch and the workspace is not
 *            used (it may be NULL); otherwise each branch runs the split-KV
 *            producer into `workspace` (ef_diff_attention_workspace_size bytes,
 *            16-byte aligned, reused by both branches) and its combine.
 * Other errors as for ef_attention_splitkv; all buffers are caller-owned and
 * the call is asynchronous on `stream`.
 */
ef_status ef_diff_attention(const void* q1, const void* q2, const void* k1, const void* k2,
                            const void* v, float* o, const float* lambda_q1,
                            const float* lambda_k1, const float* lambda_q2,
                            const float* lambda_k2, const float* norm_weight, float lambda_init,
                            float eps, int B, int Hq, int Hkv, int Sq, int Skv, int D,
                            float scale, int causal, int partition_size, void* workspace,
                            size_t workspace_bytes, void* stream);

/*
 * Workspace bytes ef_diff_attention needs for this shape and partition_size:
 * 0 when the resolved partition covers every key (single pass), else the
 * split-KV workspace of one branch. Returns 0 for invalid arguments too.
 */
size_t ef_diff_attention_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                        int partition_size);

/*
 * Decode with an output-channel split (section 7.2: at batch 1 the paper's
 * selected decode kernel gives each head two blocks that compute the same
 * scores and softmax and write different halves of the output, with no merge
 * kernel; the N parallel refinement of the p.V product, section 4.1 and table
 * "rules"). Each key
 * partition of each (batch, kv head) is evaluated by d_splits workgroups:
 * every one reads the partition's K rows and recomputes the scores, and reads,
 * accumulates and writes only its D/d_splits value channels. The output is
 * ef_attention_splitkv's.
 *   q, k, v, o, B, Hq, Hkv, Sq, Skv, D, scale, causal : as ef_attention_splitkv;
 *            at most 8 query rows per kv head ((Hq/Hkv)*Sq <= 8), else
 *            EF_ERR_INVALID_SPLIT.
 *   d_splits : 1, 2 or 4 (else EF_ERR_INVALID_SPLIT).
 *   partition_size : as ef_attention_splitkv (0 = the model's choice). When it
 *            covers every key (one partition) each workgroup writes its
 *            channels of o directly: no workspace (it may be NULL) and no
 *            merge. Otherwise the workspace (ef_attention_decode_dsplit_workspace_size
 *            bytes, 16-byte aligned, counters zero on entry and left zero, as for
 *            ef_attention_splitkv; counter slot (b*Hkv + hk)*d_splits + slice)
 *            holds the states, which every channel slice combines for its own
 *            channels (in the producer when P <= 64 and B*Hkv*d_splits <= 512).
 */
ef_status ef_attention_decode_dsplit(const void* q, const void* k, const void* v, float* o,
                                     int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                     float scale, int causal, int d_splits, int partition_size,
                                     void* workspace, size_t workspace_bytes, void* stream);

/*
 * Workspace bytes of ef_attention_decode_dsplit: 0 with one partition, else
 * the split-KV layout (the same counter region and states). 0 for invalid
 * arguments too.
 */
size_t ef_attention_decode_dsplit_workspace_size(int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                                 int d_splits, int partition_size);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc):
 * ef_attention_splitkv with the workspace replaced by a scratch array of
 * static device storage that the library holds, EF_STATIC_SCRATCH_BYTES per
 * device. The array is reserved when the library's code object is loaded on
 * a device and held until the process ends; the call itself allocates
 * nothing. The first call on a device also looks up that device's copy of
 * the array (a host-side query, not a stream operation), so make it outside
 * graph capture.
 *   Arguments, validation and output: as ef_attention_splitkv, without
 *   `workspace` and `workspace_bytes`. Returns EF_ERR_SCRATCH_TOO_SMALL, with
 *   nothing enqueued, when ef_attention_splitkv_workspace_size(...) for these
 *   arguments exceeds EF_STATIC_SCRATCH_BYTES (every other argument error is
 *   reported first), and EF_ERR_HIP when the scratch array cannot be found on
 *   the current device.
 * Every call on one device shares that device's scratch, which keeps the last
 * call's partial states: calls that overlap in time on one device race with
 * each other and must be ordered (e.g. issued on one stream). The arrival
 * counters in the scratch start at zero and every completed call leaves them
 * at zero.
 */
#define EF_STATIC_SCRATCH_BYTES ((size_t)32 << 20)

ef_status ef_attention_splitkv_noalloc(const void* q, const void* k, const void* v, float* o,
                                       int B, int Hq, int Hkv, int Sq, int Skv, int D,
                                       float scale, int causal, int partition_size,
                                       void* stream);

#ifdef __cplusplus
}
#endif

#endif /* EF_ATTENTION_H */
