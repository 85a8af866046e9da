/*
 * pdb -- sequentially-correct parallel SGD over sparse examples on one
 * MI355X (gfx950) GPU.  C ABI.
 *
 * The method (Goel, Agrawal, Chawla, Elmagarmid, "Parameter Database:
 * Data-centric Synchronization for Scalable Machine Learning"):
 *   - the sequential computation of Algorithm 1 and Definition 4 is the
 *     correctness target: iterations apply one after another, each reading
 *     the parameters it needs before writing them;
 *   - with stochastic gradient descent an iteration is one training example
 *     (Sec. 6.3) and its update is the gradient step of Sec. 2;
 *   - the read and write constraints of Sec. 4.4 only order accesses to the
 *     same parameter partition, and Theorem 2 shows that enforcing them gives
 *     the sequential result.  Here a partition is a single feature, so two
 *     examples must keep their order exactly when they share a feature, and
 *     examples that share none may run concurrently.
 *
 * pdb_schedule computes, per example, its conflict level: 1 + the largest
 * level among the earlier examples that share a feature with it (1 if
 * none).  Examples of one level touch pairwise disjoint features.
 * pdb_sgd_epoch / pdb_mf_epoch apply one epoch level by level; the result is
 * bitwise the sequential result of the fixed per-example arithmetic below.
 *
 * Conventions for every entry point:
 *   - pointers named as device pointers must point to device memory owned
 *     by the caller (e.g. allocated through PyTorch); the library never
 *     frees or keeps them past the call;
 *   - work is enqueued on the caller's stream; entry points that say
 *     "synchronous" wait for that stream before returning;
 *   - every entry point returns PDB_OK (0) or a negative pdb_status; no
 *     exception or abort crosses the ABI;
 *   - sizes: n, d, nnz < 2^31.
 *
 * Per-example arithmetic (binary32, round to nearest, subnormals kept,
 * fused multiply-add only where written as fma):
 *   entries (c_k, x_k), k = 0..m-1 in CSR order (x_k = 1 when val is NULL);
 *   partial sums p_j = 0 for j = 0..63; p_{k mod 64} = fma(w[c_k], x_k, p_{k mod 64});
 *   butterfly: for o = 1,2,4,8,16,32 every p_j becomes p_j + p_{j xor o}; z = p_0;
 *   logistic: g = 1/(1 + exp(min(-z, 87))) - (y > 0 ? 1 : 0) with one
 *   correctly rounded division (the cap keeps 1 + exp below 2^126; it only
 *   changes results for z < -87, where the logistic value is below 1.7e-38),
 *   exp by Cody-Waite reduction (k = rint(x log2 e), ln 2 split into two
 *   floats) and the degree-7 Taylor polynomial of e^r, pairs c_j + c_{j+1} r
 *   combined by Horner's rule in r^2 (p01 + r^2 (p23 + r^2 (p45 + r^2 p67))),
 *   scaled by 2^k;   least squares: g = z - y;
 *   s = lr * g;  w[c_k] = fma(-s, x_k, w[c_k]) (values read before any write).
 * Matrix completion (rank 32): q_j = fma(U_u[j], V_i[j], 0), butterfly over
 *   o = 1..16, e = r - q_0;  U_u[j] = fma(lr, e*V_i[j] - reg*U_u[j], U_u[j]),
 *   V_i[j] = fma(lr, e*U_u[j] - reg*V_i[j], V_i[j]) with the old U_u[j], V_i[j].
 */
#ifndef PDB_H
#define PDB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct ihipStream_t *hipStream_t;

typedef enum pdb_status {
    PDB_OK = 0,
    PDB_ERR_INVALID_ARG = -1, /* null pointer, negative size, unsupported rank or loss */
    PDB_ERR_BAD_CSR = -2,     /* malformed CSR (see pdb_validate_csr) */
    PDB_ERR_WORKSPACE = -3,   /* workspace pointer NULL or smaller than required */
    PDB_ERR_HIP = -4,         /* a HIP runtime call failed; pdb_last_hip_error() has the code */
    PDB_ERR_DEVICE = -5,      /* a device-side check failed (spin-wait watchdog, inconsistent schedule) */
    PDB_ERR_UNSUPPORTED = -6  /* sizes beyond 2^31 - 1, or beyond a limit an entry point states */
} pdb_status;

typedef enum pdb_loss { PDB_LOGISTIC = 0, PDB_SQUARED = 1 } pdb_loss;

typedef enum pdb_sched_method {
    PDB_SCHED_AUTO = 0,      /* chain, else spine when it applies, else the walk on chain-like
                                inputs (at most a quarter of the examples share no feature
                                with the one before them), else the short-row walk when no row
                                holds more than 4 entries, else dataflow */
    PDB_SCHED_CHAINSCAN = 1, /* chain-scan relaxation until the fixed point */
    PDB_SCHED_DATAFLOW = 2,  /* each example waits for its previous writers' levels */
    PDB_SCHED_SPINE = 3,     /* the most frequent feature's rows as a spine: applies when that
                                feature misses at most 1024 rows whose entries number at most
                                4096; otherwise dataflow runs (method_used says which) */
    PDB_SCHED_CHAIN = 4,     /* every example conflicts with the one before it: levels are
                                1..n, checked in one pass over the previous writers; otherwise
                                dataflow runs.  Auto tries this first. */
    PDB_SCHED_WALK = 5,      /* one block walks the rows in order, windows of rows staged in
                                LDS; dataflow runs instead when a row holds more than 16384
                                entries.  Under auto, when the rows form at most one run per
                                512 rows (a run: rows that each share a feature with the row
                                before) and n >= 65536, a grid settles the runs one after
                                another instead, each by a prefix maximum over its rows */
    PDB_SCHED_SHORT = 6      /* short rows (matrix completion): one block settles sub-chunks of
                                64 consecutive rows strictly in order, the waves taking turns of
                                several consecutive sub-chunks, each sub-chunk by as many rounds
                                of lane shuffles as its longest chain of in-sub-chunk writers,
                                with the levels of the last 256 sub-chunks kept in an LDS ring;
                                dataflow runs instead when a row holds more than 4 entries */
} pdb_sched_method;
/* Two dataflow forms.  The wave-per-example form runs when the chain check
 * ran (PDB_SCHED_AUTO or PDB_SCHED_CHAIN), found the input not chain-like
 * (more than a quarter of the examples share no feature with the one before
 * them) and rows hold at least 16 entries on average.  Every other dataflow
 * run, an explicit PDB_SCHED_DATAFLOW request among them, uses the batch form
 * (64-example batches per wave). */

/* Which execution pdb_sgd_epoch, pdb_mf_epoch and pdb_batch_epoch use. */
typedef enum pdb_epoch_mode {
    PDB_EPOCH_AUTO = 0,     /* sync-free when it is possible and levels are wide on average
                               (n >= 8 L, L from pdb_levels.L_host), else level by level;
                               mini-batches: sync-free whenever it is possible */
    PDB_EPOCH_LEVELS = 1,   /* level by level */
    PDB_EPOCH_SYNCFREE = 2  /* sync-free when possible (prev_nz set, workspace large enough) */
} pdb_epoch_mode;

/* Which execution pdb_stale_epoch uses. */
typedef enum pdb_stale_mode {
    PDB_STALE_AUTO = 0,      /* windowed on chain-like inputs whose windows fit, else sync-free */
    PDB_STALE_SYNCFREE = 1,
    PDB_STALE_WINDOWED = 2   /* windowed wherever the windows fit */
} pdb_stale_mode;

/* Execution options.  Every option selects among executions that give
 * bitwise the same result, or bounds a device-side wait; none changes what is
 * computed.  A NULL pointer means all defaults; otherwise fill the struct with
 * pdb_options_init and change fields.  Options act only on the call they are
 * passed to: the library keeps no configuration between calls and reads no
 * environment variables. */
typedef struct pdb_options {
    int32_t epoch_mode;            /* pdb_epoch_mode (default PDB_EPOCH_AUTO) */
    int32_t pipeline;              /* level-by-level epoch: 1 runs of narrow levels go through the
                                      one-block pipeline (default), 0 every level on the plain path */
    int32_t pipeline_width;        /* widest level a pipeline run may include (>= 1, default 4);
                                      when no level is wider, the whole epoch is one pipeline run
                                      over the examples in index order (the same result) */
    int32_t thin_max;              /* widest level run by one block alone (>= 1, default 16) */
    int64_t hot_features;          /* cap on the weights the pipeline caches in LDS; -1 (default)
                                      all that fit */
    int64_t spin_timeout_us;       /* watchdog of every device-side wait, in microseconds (default
                                      20,000,000): a wait that lasts longer gives up, every kernel
                                      of the call exits, and the call (or pdb_workspace_status)
                                      reports PDB_ERR_DEVICE.  0 gives up on any wait not met
                                      within a few polls, which exercises that path */
    int32_t batch_thin_max;        /* level-by-level mini-batch epoch: widest batch level run by
                                      one block alone (>= 1, default 2) */
    int32_t batch_syncfree_blocks; /* sync-free mini-batch epoch: blocks in flight (>= 1,
                                      default 32; at most one per compute unit) */
    int32_t stale_mode;            /* pdb_stale_mode (default PDB_STALE_AUTO) */
    int32_t dense_stream;          /* pdb_dense_gd: 1 streams the tiles from memory even when they
                                      fit in LDS, 0 (default) keeps them resident when they fit */
    int32_t mf_one_cu;             /* sync-free pdb_mf_epoch: 1 runs every rating on one compute
                                      unit (hand-overs through its LDS and L1 cache), 0 spreads the
                                      ratings over the device (device-scope hand-overs), -1
                                      (default) one compute unit when levels are narrow (n < 16 L)
                                      and (n_users + n_items) * 256 <= 2^32 (the words are
                                      addressed with 32-bit byte offsets); 1 falls back to the
                                      device-wide execution when they do not fit that bound */
} pdb_options;

/* Fills *opt with the defaults above.  Host only. */
int pdb_options_init(pdb_options *opt);

/* Sparse examples in CSR form (Definition 1: the immutable data set D). */
typedef struct pdb_csr {
    const int64_t *row_ptr; /* device, [n+1]; row_ptr[0] = 0, non-decreasing */
    const int32_t *col;     /* device, [nnz]; within a row strictly increasing, in [0, d) */
    const float *val;       /* device, [nnz]; NULL means every stored value is 1.0f */
    int64_t nnz;            /* = row_ptr[n] */
} pdb_csr;

/* Output of pdb_schedule (all device arrays owned by the caller). */
typedef struct pdb_levels {
    int32_t *level;     /* [n]   conflict level of each example, 1-based */
    int32_t *perm;      /* [n]   examples ordered by (level, index) */
    int64_t *level_ptr; /* [n+1] level l holds perm[level_ptr[l-1] .. level_ptr[l]), l = 1..L;
                                 level_ptr[0] = 0, level_ptr[L] = n */
    int32_t *n_levels;  /* [1]   L */
    int32_t *prev_nz;   /* [nnz] or NULL: for each stored entry, the CSR index of the previous
                                 entry (earlier example) on the same feature, -1 if none */
    /* host-side summary written by pdb_schedule; zero means unknown */
    int64_t L_host;         /* L */
    int64_t max_width_host; /* largest level width */
} pdb_levels;

/* Optional host-side report of pdb_schedule. */
typedef struct pdb_schedule_info {
    int32_t method_used;  /* pdb_sched_method that produced the levels */
    int32_t rounds;       /* chain-scan rounds, or spine solver rounds */
    int64_t n_levels;     /* L */
    int64_t max_width;    /* largest level width */
} pdb_schedule_info;

/* Human-readable text for a pdb_status code (static storage). */
const char *pdb_strerror(int status);

/* hipError_t of the last failing HIP call in this thread (0 if none). */
int pdb_last_hip_error(void);

/* Device workspace (bytes) needed by pdb_schedule, pdb_transpose and
 * pdb_prev_writer for these sizes.  Host-only arithmetic. */
int pdb_schedule_workspace_bytes(int64_t n, int64_t d, int64_t nnz, size_t *bytes);

/* Device workspace (bytes) for pdb_sgd_epoch with d features, or for
 * pdb_mf_epoch with d = (n_users + n_items) * rank; d = 0 for pdb_validate_csr,
 * pdb_workspace_status and pdb_check_reciprocal.  Host-only arithmetic.  A
 * workspace of this size lets pdb_sgd_epoch run sync-free. */
int pdb_epoch_workspace_bytes(int64_t d, size_t *bytes);

/* Conflict levels (read/write constraints of Sec. 4.4 at feature grain,
 * Theorem 2): fills levels->level, perm, level_ptr, n_levels, prev_nz (when
 * not NULL) and the host fields L_host, max_width_host.  labels is accepted
 * for symmetry with pdb_sgd_epoch and ignored: conflicts depend only on the
 * sparsity pattern.  ws: device workspace of at least
 * pdb_schedule_workspace_bytes().  opt: only spin_timeout_us applies (the
 * dataflow and short-row methods wait on device).  Synchronous (it waits
 * for the stream); a device-side wait that gave up returns PDB_ERR_DEVICE.
 * Does not check the CSR: call pdb_validate_csr first on untrusted input. */
int pdb_schedule(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                 pdb_levels *levels, int method, pdb_schedule_info *info, void *ws,
                 size_t ws_bytes, const pdb_options *opt, hipStream_t stream);

/* One SGD epoch over all n examples in place on w (device, [d]), with the
 * per-example arithmetic stated at the top of this header, for loss
 * PDB_LOGISTIC (labels y in {-1,+1}: target y > 0) or PDB_SQUARED.  levels
 * must come from pdb_schedule on the same CSR (or be an equivalent
 * grouping: every level's examples pairwise feature-disjoint, every
 * conflicting pair in index order across levels).  Two executions, bitwise
 * the same result:
 *   - level by level (narrow levels: a width-1 run is one dependent chain);
 *   - sync-free, the Read Protocol of Sec. 5 at feature grain: examples in
 *     index order, each entry waiting only until its feature was written by
 *     its previous writer (levels->prev_nz), no barriers.  The examples are
 *     dealt to the waves of a cooperatively launched grid in turn (every
 *     block resident, so the earliest unfinished example always runs; a
 *     refused launch returns PDB_ERR_HIP).  Chosen when
 *     n >= 8 L, levels->prev_nz is set and ws_bytes covers
 *     pdb_epoch_workspace_bytes(d) (opt->epoch_mode forces levels or, where
 *     possible, sync-free).
 * ws: at least pdb_epoch_workspace_bytes(0).  Asynchronous; a device error
 * (watchdog) is reported by pdb_workspace_status on ws. */
int pdb_sgd_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d, float *w,
                  float lr, int loss, const pdb_levels *levels, void *ws, size_t ws_bytes,
                  const pdb_options *opt, hipStream_t stream);

/* For callers that cannot allocate device memory (code under stream capture,
 * tight serving loops, hosts that forbid allocation): pdb_sgd_epoch with the
 * workspace replaced by a scratch array the library holds in device memory
 * of each GPU it runs on (the control block and one 8-byte word per feature,
 * 16 MiB + 512 bytes, kept until the process ends).  Same arguments, result
 * and executions as pdb_sgd_epoch; d at most 2^21 (2,097,152), else
 * PDB_ERR_UNSUPPORTED.  It calls no allocating routine.  status: device,
 * [1], or NULL: after the epoch a kernel on the stream writes 0 there, or a
 * nonzero device error code (watchdog) -- the report pdb_workspace_status
 * gives for pdb_sgd_epoch.  Every call on one GPU uses that GPU's scratch:
 * calls that overlap on one GPU (other streams, other threads) race and must
 * be ordered by the caller.  Asynchronous. */
int pdb_sgd_epoch_noalloc(const pdb_csr *csr, const float *labels, int64_t n, int64_t d,
                          float *w, float lr, int loss, const pdb_levels *levels, int32_t *status,
                          const pdb_options *opt, hipStream_t stream);

/* One matrix-completion SGD epoch (rank 32).  Rating t's loss is Eq. 2's
 * squared error with its L2 regulariser on the two factor rows it touches,
 * (r_t - <U_u, V_i>)^2 / 2 + reg (|U_u|^2 + |V_i|^2) / 2, and its update is
 * the gradient step of Sec. 2 on that loss (the per-rating arithmetic at the
 * top of this header; both rows from their values before the step).  Rating
 * t touches user row U[user[t]] (device [n_users*32]) and item row
 * V[item[t]] (device [n_items*32]); levels from pdb_schedule on the CSR whose
 * row t is {user[t], n_users + item[t]}.  Runs level by level or sync-free
 * (the sync-free run needs levels->prev_nz and
 * pdb_epoch_workspace_bytes((n_users + n_items) * 32)); under
 * PDB_EPOCH_AUTO sync-free when levels are wide (n >= 8 L) or when the
 * one-compute-unit execution applies (pdb_options.mf_one_cu), else level by
 * level.  Every execution gives bitwise the same U and V.  Asynchronous. */
int pdb_mf_epoch(const int32_t *user, const int32_t *item, const float *rating, int64_t n,
                 float *U, int64_t n_users, float *V, int64_t n_items, int32_t rank, float lr,
                 float reg, const pdb_levels *levels, void *ws, size_t ws_bytes,
                 const pdb_options *opt, hipStream_t stream);

/* Checks row_ptr[0] == 0, row_ptr non-decreasing, row_ptr[n] == nnz, every
 * column in [0, d) and strictly increasing within its row.  Synchronous.
 * Returns PDB_OK or PDB_ERR_BAD_CSR.  ws: pdb_epoch_workspace_bytes(). */
int pdb_validate_csr(const pdb_csr *csr, int64_t n, int64_t d, void *ws, size_t ws_bytes,
                     hipStream_t stream);

/* Checks that levels are a schedule the epoch may run (Theorem 2 with the
 * read/write constraints of Sec. 4.4 at feature grain):
 *   - level_ptr[0] = 0, non-decreasing, level_ptr[L] = n with L = *n_levels
 *     (1 <= L <= n when n > 0), and perm a permutation of 0..n-1 with
 *     level[perm[e]] = l for every e in [level_ptr[l-1], level_ptr[l]);
 *   - along every feature's occurrences in example order the levels strictly
 *     increase: each example's level exceeds that of the latest earlier
 *     example sharing a feature with it.  That makes every level's examples
 *     pairwise feature-disjoint and puts every conflicting earlier example in
 *     a lower level;
 *   - when levels->prev_nz is set, it equals the previous writers computed
 *     here from the CSR.
 * The previous writers are recomputed from the CSR (the transpose of
 * pdb_schedule), so nothing in levels is trusted.  ws: at least
 * pdb_schedule_workspace_bytes(n, d, nnz).  Synchronous.  Returns PDB_OK, or
 * PDB_ERR_DEVICE when a check fails (and writes nothing).  Does not check the
 * CSR: call pdb_validate_csr first on untrusted input. */
int pdb_validate_schedule(const pdb_csr *csr, int64_t n, int64_t d, const pdb_levels *levels,
                          void *ws, size_t ws_bytes, hipStream_t stream);

/* Waits for the stream, then returns PDB_ERR_DEVICE if a kernel that used
 * ws recorded a device-side failure (and clears it), else PDB_OK. */
int pdb_workspace_status(void *ws, hipStream_t stream);

/* Mini-batches (Sec. 6.3: gradient descent with a fixed batch of examples per
 * iteration).  Batch b is examples [b*B, min((b+1)*B, n)), nb = ceil(n/B);
 * its parameter set is the union of its examples' features.  Device arrays
 * owned by the caller, written by pdb_batch_schedule:
 *   bptr    [nb+1]   batch b's union entries are u in [bptr[b], bptr[b+1]);
 *   ucol    [nnz]    feature of union entry u, ascending within a batch
 *                    (the first U entries are used);
 *   uptr    [nnz+1]  union entry u's occurrences are occ[uptr[u] .. uptr[u+1]);
 *   occ     [nnz]    CSR entry indices ordered by (batch, feature, index);
 *   occ_row [nnz]    the example of each of them;
 *   occ_u   [nnz]    the union entry of each of them;
 *   unext   [nnz]    NULL, or the next union entry on the same feature (-1 if
 *                    none; written when levels->prev_nz is set): the
 *                    sync-free epoch publishes what the next batch needs
 *                    first. */
typedef struct pdb_batches {
    int64_t *bptr;
    int32_t *ucol;
    int64_t *uptr;
    int32_t *occ;
    int32_t *occ_row;
    int32_t *occ_u;
    int32_t *unext;
    int64_t U_host; /* union size U, written by pdb_batch_schedule */
} pdb_batches;

/* Conflict levels of mini-batches of `batch` examples (1 <= batch <= 4096):
 * fills *batches, then runs pdb_schedule on the CSR whose rows are the
 * batches (row_ptr = bptr, col = ucol), so levels describe the nb batches:
 * level [nb], perm [nb] (batch indices), level_ptr [nb+1], and prev_nz (when
 * not NULL) over the U union entries.  Two batches conflict when they share
 * a feature (Sec. 4.4 at feature grain); batches of one level are pairwise
 * feature-disjoint.  With batch = 1 the levels are those of pdb_schedule.
 * ws: at least pdb_schedule_workspace_bytes(n, d, nnz).  Synchronous. */
int pdb_batch_schedule(const pdb_csr *csr, int64_t n, int64_t d, int64_t batch,
                       pdb_batches *batches, pdb_levels *levels, int method,
                       pdb_schedule_info *info, void *ws, size_t ws_bytes,
                       const pdb_options *opt, hipStream_t stream);

/* One epoch of mini-batch gradient descent in place on w (device, [d]).
 * Batch b, in the sequential order of batches: every example i of b computes
 * z_i and s_i = lr * g_i with the per-example arithmetic at the top of this
 * header against the weights as they were when b started (all reads before
 * any write, Definition 3); then each feature f of b takes, in example
 * order, w_f = fma(-s_i, x_if, w_f) -- the gradient step of Sec. 2 on the
 * sum of the batch's losses.  With batch = 1 this is pdb_sgd_epoch's
 * result.  batches and levels from pdb_batch_schedule with the same batch.
 * Two executions, bitwise the same result, one block per batch:
 *   - batch levels in order, a level's batches concurrently (Theorem 2);
 *   - sync-free (the Read Protocol of Sec. 5 with a batch as the iteration):
 *     batches in index order, each waiting only until each of its features
 *     was written by its previous writer (levels->prev_nz over the union
 *     entries), no barriers.  Chosen when levels->prev_nz is set and ws_bytes
 *     covers pdb_epoch_workspace_bytes(d) (opt->epoch_mode = PDB_EPOCH_LEVELS forces
 *     batch levels).
 * ws: at least pdb_epoch_workspace_bytes(0).  Asynchronous; a device error
 * (watchdog) is reported by pdb_workspace_status on ws. */
int pdb_batch_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d, int64_t batch,
                    float *w, float lr, int loss, const pdb_batches *batches,
                    const pdb_levels *levels, void *ws, size_t ws_bytes,
                    const pdb_options *opt, hipStream_t stream);

/* Device workspace (bytes) for pdb_stale_epoch: the control block, one
 * 64-bit word and three ints per stored entry.  Host-only arithmetic. */
int pdb_stale_workspace_bytes(int64_t nnz, size_t *bytes);

/* One epoch of bounded-delay SGD (Sec. 7: the Asynchronous Read Constraint
 * lets iteration alpha read a partition once the write of iteration
 * alpha - 1 - delay is done), in the execution that reads as early as that
 * allows: example alpha computes z, with the per-example arithmetic at the
 * top of this header, from the values its features had after examples
 * 0 .. alpha - delay - 1 (the initial w where no such example wrote them);
 * each example's update is then applied in example order to each of its
 * features, w_f = fma(-s, x, w_f), on the value the previous writer left.
 * delay = 0 is pdb_sgd_epoch's result; delay >= n - 1 reads the initial
 * weights everywhere (pdb_batch_epoch with batch = n).  prev_nz: device,
 * [nnz], from pdb_schedule on the same CSR.  Finding each entry's read
 * source takes up to `delay` steps back along its feature.  Two executions,
 * bitwise the same result:
 *   - windowed, one block: examples in windows of delay + 1, whose reads all
 *     come from earlier windows; chosen when every window holds at most 2048
 *     examples and 2048 stored entries and at most a quarter of the examples
 *     share no feature with the example before them (opt->stale_mode forces
 *     the sync-free execution, or the windowed one where windows fit);
 *   - sync-free: examples in index order, each waiting on the words of its
 *     read sources and previous writers (dealt to the waves of a
 *     cooperatively launched grid in turn, as in pdb_sgd_epoch).
 * ws: at least pdb_stale_workspace_bytes(nnz).  Synchronous: it reads back
 * the largest window's size to choose; a device error (watchdog) is reported
 * by pdb_workspace_status on ws. */
int pdb_stale_epoch(const pdb_csr *csr, const float *labels, int64_t n, int64_t d, float *w,
                    float lr, int loss, int64_t delay, const int32_t *prev_nz, void *ws,
                    size_t ws_bytes, const pdb_options *opt, hipStream_t stream);

/* Dense full-batch gradient descent (the update of Sec. 2 with every example
 * in every iteration; the dense linear-regression workloads of Sec. 6.1-6.2).
 *
 * The work is split over an R x C grid of workers: rows in blocks of
 * row_block, columns in blocks of col_block (a multiple of 4), R =
 * ceil(n / row_block), C = ceil(d / col_block).  The blocking fixes the
 * summation order, so pdb_dense_plan is deterministic: it picks the blocks
 * for `workers` workers (<= 0: the current device's compute units), with
 * C / R near sqrt(d / n).  Host-only arithmetic apart from the device query.
 * PDB_ERR_UNSUPPORTED when a block would exceed 4096 rows or 16384 columns. */
int pdb_dense_plan(int64_t n, int64_t d, int workers, int64_t *row_block, int64_t *col_block);

/* Device workspace (bytes) for pdb_dense_gd: the control block and two
 * buffers of 64-bit words, 2 C n partial dot products and 2 R d partial
 * gradients.  Host-only arithmetic. */
int pdb_dense_workspace_bytes(int64_t n, int64_t d, int64_t row_block, int64_t col_block,
                              size_t *bytes);

/* `iters` iterations of full-batch gradient descent in place on w (device,
 * [d]).  X: device, n x d, row-major with row stride ldx >= d (16-byte
 * alignment and ldx % 4 == 0 take the vector loads; any layout works).
 * labels: device, [n].  One iteration, every z_i from the weights before it:
 *   z_i = <X_i, w>;  s_i = lr * g(z_i, y_i) with g as at the top of this
 *   header;  G_j = sum_i s_i X_ij;  w_j = w_j - G_j.
 * Summation order: within a column block, column k (k from 0 at the block
 * start) goes to partial sum floor(k / 4) mod 64 as fma(X_ik, w_k, p), then
 * the butterfly as at the top of this header; z_i adds the column blocks'
 * results in block order (starting from block 0's).  A row block's partial
 * of G_j adds, in order (starting from the first's), the partials of its
 * chunks of 32 rows, each fma(s_i, X_ij, p) over the chunk's rows in order
 * from 0; G_j adds the row blocks' partials in block order.  The tile of a
 * worker stays in LDS across iterations when col_block + row_block (rounded
 * up to 4) + row_block col_block floats, plus room for its staged partials,
 * fit 36864 floats (unless opt->dense_stream is set); otherwise it is read
 * from memory twice per iteration.  Worker (r, c) waits only for the
 * partials of its row group and of its column group (the read constraint of
 * Sec. 4.4 per partition), never on a grid-wide barrier; the R C workers
 * must be resident at once (one per compute unit; PDB_ERR_UNSUPPORTED
 * otherwise).  Nothing changes when n, d or iters is 0.
 * ws: at least pdb_dense_workspace_bytes(n, d, row_block, col_block).
 * Asynchronous; a device error (watchdog) is reported by pdb_workspace_status
 * on ws. */
int pdb_dense_gd(const float *X, int64_t ldx, const float *labels, int64_t n, int64_t d,
                 float *w, float lr, int loss, int64_t iters, int64_t row_block,
                 int64_t col_block, void *ws, size_t ws_bytes, const pdb_options *opt,
                 hipStream_t stream);

/* Per-feature occurrence lists (the transpose that exposes which examples
 * share a feature): col_ptr (device, [d+1]) and csc_row (device, [nnz],
 * rows ascending within a feature).  ws as for pdb_schedule.  Synchronous. */
int pdb_transpose(const pdb_csr *csr, int64_t n, int64_t d, int64_t *col_ptr, int32_t *csc_row,
                  void *ws, size_t ws_bytes, hipStream_t stream);

/* Previous writer of every stored entry (the per-feature version the Read
 * Protocol of Sec. 5 waits for): prev_row (device, [nnz]) = the latest
 * earlier example touching the same feature, -1 if none; prev_nz (device,
 * [nnz], may be NULL) = the CSR index of that example's entry.  ws as for
 * pdb_schedule.  Synchronous. */
int pdb_prev_writer(const pdb_csr *csr, int64_t n, int64_t d, int32_t *prev_row,
                    int32_t *prev_nz, void *ws, size_t ws_bytes, hipStream_t stream);

/* Self-check of the division in the logistic step on this device: for every
 * binary32 b whose bit pattern lies in [lo_bits, hi_bits) (within
 * [0x3F800000, 0x7E800000), i.e. 1 <= b < 2^126, the range of 1 + exp above),
 * compares the kernels' reciprocal of b with the IEEE quotient 1/b.  Writes
 * the number of mismatches and the smallest mismatching bit pattern
 * (0xFFFFFFFF if none) to host memory.  ws: pdb_epoch_workspace_bytes().
 * Synchronous. */
int pdb_check_reciprocal(uint32_t lo_bits, uint32_t hi_bits, uint64_t *mismatches,
                         uint32_t *first_bad, void *ws, size_t ws_bytes, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PDB_H */
