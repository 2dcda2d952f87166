/*
 * libargus: MI355X (gfx950) kernels for the data-parallel hot path of ARGUS
 * ("ARGUS: Production-Scale Tracing and Performance Diagnosis for over
 * 10,000-GPU Clusters", arXiv 2606.20374).
 *
 *   argus_summarize     raw per-rank kernel-event arrays -> per (rank, step,
 *                       kernel id) count, sum, min, max and octave histogram
 *                       of durations, plus per (rank, step) aggregates
 *                       (section 4.3 record fields; section 5.2 grouping per
 *                       kernel and rank in each window, log-duration grid).
 *   argus_cross_rank    summaries -> per (step, kernel) robust cross-rank
 *                       statistics (lower median, quartiles, MAD), per-cell
 *                       robust z, outlier / IQR-fence / degraded-pair flags
 *                       and per (rank, step) straggler decisions (section
 *                       6.2 and Eq. 4; z-score of Appendix B).
 *   argus_iter_windows  per-rank step times -> L1 jitter windows, effective
 *                       width, change point and class (section 6.1,
 *                       Appendix B).
 *   argus_kde           raw events + their summaries -> per (rank, step,
 *                       kernel id) duration clusters from the valleys of a
 *                       Gaussian KDE over log-duration, each reported as
 *                       (count, p50, p99) (section 5.2, Eq. 1).
 *   argus_w1            clusters -> per (step, kernel) cross-rank
 *                       Wasserstein-1 deviation scores of the reconstructed
 *                       lognormal-mixture CDFs and the IQR upper fence over
 *                       them (section 6.2, Eq. 2 - 4).
 *   argus_l2            summaries + a routing table and parallelism groups ->
 *                       per (step, event, group) mean, sample std, CV class
 *                       and per-rank z-score straggler flags, every event
 *                       compared only inside the groups of its dimension
 *                       (section 6.1, Table "routing"; Appendix B, Eq. 5).
 *
 * Conventions for every entry point:
 *   - All array pointers are DEVICE pointers owned by the caller. The library
 *     never allocates or frees device memory; calls that need scratch take a
 *     caller workspace whose size the matching *_workspace query reports.
 *   - Calls are asynchronous on the caller's stream (a hipStream_t passed as
 *     void*; NULL is the default stream). Results are visible after the
 *     caller synchronises that stream.
 *   - The return value is a status checked on the host before any launch
 *     (ARGUS_E*); nothing is launched when it is not ARGUS_OK. Conditions
 *     that only the device can see (malformed segment offsets, out-of-range
 *     step times) are OR-ed as ARGUS_DEV_* bits into the optional device
 *     word *dev_status, which the call first resets to 0.
 *   - The library writes every element of every non-NULL output, including
 *     identity values for empty cells, so outputs need no pre-clearing. The
 *     one exception is argus_summarize (and _keyed): for an absent cell
 *     (count 0) only the count is written, see there.
 *   - Calls keep no mutable global state and are safe from several host
 *     threads on different streams.
 *   - Integer outputs are exact and deterministic; float outputs are
 *     computed in double and rounded once to float (argus_w1 reports its
 *     doubles unrounded).
 */
#ifndef ARGUS_H
#define ARGUS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ARGUS_ABI_VERSION 1
#define ARGUS_NBINS 32          /* octave bins per cell */
#define ARGUS_MAX_KERNELS 65536 /* n_kernels limit */
#define ARGUS_MAX_STREAMS 64    /* n_streams limit */
#define ARGUS_MAX_XR_RANKS 16384 /* argus_cross_rank: n_ranks limit */
#define ARGUS_MAX_XR_KERNELS 16384 /* argus_cross_rank: n_kernels limit */
#define ARGUS_MAX_L1_STEPS 4096  /* argus_iter_windows: n_steps limit */
#define ARGUS_MAX_KDE_KERNELS 16384 /* argus_kde: n_kernels limit */
#define ARGUS_KDE_MAXC 4         /* argus_kde: clusters reported per cell */
#define ARGUS_MAX_W1_RANKS 16384 /* argus_w1: n_ranks limit */
#define ARGUS_MAX_W1_GRID 2048   /* argus_w1: grid points limit */
#define ARGUS_MAX_W1_STEPS 65535 /* argus_w1: n_steps limit */
#define ARGUS_MAX_L2_RANKS 65536 /* argus_l2: n_ranks limit */
#define ARGUS_MAX_L2_DIMS 16     /* argus_l2: parallelism dimensions limit */
#define ARGUS_NOALLOC_SCRATCH_BYTES 256 /* argus_summarize_noalloc: static scratch per device */

enum {
  ARGUS_OK = 0,
  ARGUS_EINVAL = -1,      /* NULL pointer, bad dimension, bad parameter, workspace too small */
  ARGUS_EUNSUPPORTED = -2, /* current device is not gfx950 */
  ARGUS_EHIP = -3,        /* a HIP launch failed */
  ARGUS_EDEVICE = -4      /* not returned by calls; names the dev_status channel */
};

/* device-detected condition bits OR-ed into *dev_status */
enum {
  ARGUS_DEV_BAD_SEGMENT = 1, /* some seg_off range was malformed; that segment was summarized as empty */
  ARGUS_DEV_L1_DOMAIN = 2,   /* some rank had a step time outside [0, 2^40) ns; that rank got class 0x80 */
  ARGUS_DEV_KDE_SUMMARY = 4, /* argus_kde: the summaries passed in do not match the events (counts, min or
                                max); the affected cells report 0 clusters */
  ARGUS_DEV_W1_INPUT = 8,    /* argus_w1: some cell had more than ARGUS_KDE_MAXC clusters, or clusters of total
                                count 0; such cells take no part */
  ARGUS_DEV_GROUPS_MALFORMED = 16, /* argus_l2: a group range outside [0, n_ranks] or reversed (group skipped), or
                                      a member id outside [0, n_ranks) (member skipped) */
  ARGUS_DEV_GROUPS_DUPLICATE = 32, /* argus_l2: a rank listed more than once in one dimension (only its first
                                      listing counts) */
  ARGUS_DEV_L2_DOMAIN = 64,        /* argus_l2: a mean duration at or above 2^40 ns (that cell is left out) */
  ARGUS_DEV_COMPACT_CAPACITY = 128, /* argus_compact: the records did not all fit in the caller's buffer */
  ARGUS_DEV_SUMMARY_STALLED = 256   /* argus_summarize: a bounded wait inside the kernel expired in every one of
                                       its redo passes over some segment (never expected: it means a defect in
                                       the library or the device); that segment's cells may be incomplete */
};

int argus_abi_version(void);
const char* argus_status_string(int status);

/* ---------------------------------------------------------------- summarize
 *
 * Events are structure-of-arrays, grouped into n_ranks * n_steps segments:
 * segment g = r * n_steps + s covers events [seg_off[g], seg_off[g+1]).
 * Order within a segment is arbitrary. Total events may exceed 2^31.
 *
 * An event is valid iff 0 <= kernel_id < n_kernels, 0 <= stream < n_streams,
 * start_ns >= 0 and end_ns >= start_ns. Invalid events are only counted in
 * n_invalid (the paper's collectors drop under backpressure rather than mix
 * bad records in: Appendix A). For a valid event d = end_ns - start_ns and its
 * octave bin is 0 for d < 2, else min(floor(log2 d), 31).
 *
 * A segment is malformed unless 0 <= seg_off[g] <= seg_off[g+1] <= n_events
 * and its length is below 2^32; a malformed segment is summarized as empty
 * and ARGUS_DEV_BAD_SEGMENT is raised. Sums wrap modulo 2^64.
 *
 * Written cells: count is written for every cell. sum_ns, min_ns, max_ns and
 * hist are written only for present cells (count >= 1); for an absent cell
 * they keep whatever the buffers held (a caller that wants the identity
 * values 0 / INT64_MAX / INT64_MIN / 0 fills them beforehand). Large, sparse
 * key spaces (most kernel ids absent from a rank-step) thus cost 4 bytes per
 * absent cell instead of 156. Every consumer in this library (cross-rank, L2,
 * KDE, compaction) reads a cell's other fields only when its count is >= 1.
 */
typedef struct argus_events {
  const int32_t* kernel_id; /* [n_events] */
  const int32_t* stream;    /* [n_events] */
  const int64_t* start_ns;  /* [n_events] */
  const int64_t* end_ns;    /* [n_events] */
  const int64_t* seg_off;   /* [n_ranks * n_steps + 1] */
  int64_t n_events;         /* length of the four event arrays */
  int32_t n_ranks, n_steps, n_kernels, n_streams;
} argus_events_t;

typedef struct argus_summary {
  /* per cell, [n_ranks][n_steps][n_kernels] (hist: [..][ARGUS_NBINS]) */
  uint32_t* count;  /* valid events of the kernel (every cell) */
  int64_t* sum_ns;  /* sum of d (present cells only) */
  int64_t* min_ns;  /* min d (present cells only) */
  int64_t* max_ns;  /* max d (present cells only) */
  uint32_t* hist;   /* octave histogram of d (present cells only) */
  /* per segment, [n_ranks][n_steps] */
  uint32_t* n_valid;
  uint32_t* n_invalid;
  int64_t* t_first;        /* min start of valid events, INT64_MAX when none */
  int64_t* t_last;         /* max end of valid events, INT64_MIN when none */
  int64_t* step_ns;        /* t_last - t_first, 0 when no valid event */
  int64_t* busy_ns;        /* sum of d over valid events */
  int64_t* stream_busy_ns; /* [n_ranks][n_steps][n_streams] sum of d per stream */
  int64_t* wire_bytes;     /* optional (may be NULL): bytes of the uploaded summary records:
                              sum over cells with count > 0 of 33 + 5 * (nonzero bins) */
  int32_t* dev_status;     /* optional (may be NULL) */
} argus_summary_t;

/* Bytes of caller workspace argus_summarize needs (a small, fixed amount:
 * the work-queue counter of its persistent workgroups). The workspace must be
 * device memory, 4-byte aligned, and not shared by calls that may overlap. */
size_t argus_summarize_workspace(const argus_events_t* ev);

/* Every output pointer except wire_bytes and dev_status is required; hist
 * must be 16-byte aligned. workspace: see argus_summarize_workspace. */
int argus_summarize(const argus_events_t* ev, const argus_summary_t* out, void* workspace, size_t workspace_bytes,
                    void* stream);

/* For callers that cannot allocate device memory or pass a workspace (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): argus_summarize with its scratch, the work-queue counter of
 * its persistent workgroups, in a static device array of
 * ARGUS_NOALLOC_SCRATCH_BYTES that the library holds on each device it runs
 * on until the process ends. Arguments, outputs and status codes are those
 * of argus_summarize; the call allocates nothing and frees nothing. It
 * returns ARGUS_EINVAL when the call would need more scratch than the array
 * holds (argus_summarize_workspace(ev) > ARGUS_NOALLOC_SCRATCH_BYTES). Every
 * call on a device shares that device's array and resets it on its stream
 * before use: calls that may overlap on one device (other streams, other
 * host threads) race and must not be issued. */
int argus_summarize_noalloc(const argus_events_t* ev, const argus_summary_t* out, void* stream);

/* As argus_summarize, but cells are keyed by (kernel id, stream), the
 * grouping key of section 5.2: cells are [n_ranks][n_steps][n_kernels]
 * [n_streams] (cell index (g * n_kernels + kernel_id) * n_streams + stream),
 * n_kernels * n_streams <= ARGUS_MAX_KERNELS. Per-segment outputs and
 * wire_bytes are as for argus_summarize. */
int argus_summarize_keyed(const argus_events_t* ev, const argus_summary_t* out, void* workspace,
                          size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ compact
 *
 * The uploaded summary (section 5.2: only compact statistics leave the host;
 * section 8.3 compares their size with the raw trace): the present cells
 * (count >= 1) of dense summaries, every segment in order and every cell in
 * key order, as little-endian records
 *   key u32    the kernel id; with (kernel, stream) keys kid | stream << 24
 *   count u32, sum i64, min i64, max i64
 *   nnz u8     number of nonzero octave bins
 *   nnz x (bin u8, count u32) in ascending bin order
 * i.e. 33 + 5 nnz bytes (the wire_bytes of argus_summarize, per segment).
 * seg_byte_off[g] is the first byte of segment g and seg_byte_off[n_seg]
 * the total, whatever the capacity; a record is written only if it lies
 * entirely inside out[0, capacity) (else ARGUS_DEV_COMPACT_CAPACITY), so a
 * call with capacity 0 only sizes the stream. Placement is deterministic.
 */
size_t argus_compact_workspace(int32_t n_ranks, int32_t n_steps);

/* sum: count, sum_ns, min_ns, max_ns and hist (16-byte aligned) of an
 * argus_summarize (n_streams = 0, n_cells = n_kernels) or
 * argus_summarize_keyed (n_streams = NS, n_cells = n_kernels * NS) output.
 * seg_byte_off: [n_ranks * n_steps + 1]. out may be NULL when capacity = 0.
 * The workspace must be 8-byte aligned. */
int argus_compact(const argus_summary_t* sum, int32_t n_ranks, int32_t n_steps, int32_t n_cells, int32_t n_streams,
                  uint8_t* out, int64_t capacity, int64_t* seg_byte_off, int32_t* dev_status, void* workspace,
                  size_t workspace_bytes, void* stream);

/* --------------------------------------------------------------- cross-rank
 *
 * For each step s and kernel k, over the ranks r where count > 0 ("present"):
 *   x_r = min(floor((uint64)sum / count), INT64_MAX)    exact integer mean
 *   n   = number of present ranks
 * If n < min_ranks the kernel is not evaluated: med = mad = q1 = q3 = -1,
 * xmean = 0, and its cells get z = 0, flags = 0. Otherwise, with v = sorted x:
 *   med = v[(n-1)/2], q1 = v[(n-1)/4], q3 = v[3(n-1)/4]   (lower nearest-rank)
 *   mad = lower median of |x_r - med|,  madf = max(mad, 1)
 *   xmean = (float)((double)(exact sum of x) / n)
 * Per present cell of an evaluated kernel (flags bit2 = 1):
 *   z     = (float)((double)(x - med) / (1.4826 * madf))
 *   bit0  = count >= c_min_pair && 1000 (x - med) > k_mad_pm * madf && 1000 x >= ratio_pm * med
 *   bit1  = 1000 (x - q3) > alpha_pm * max(q3 - q1, 1)              (Eq. 4 upper fence)
 * Per (rank, step), over E = evaluated present kernels with med >= 1:
 *   score_pm = lower median of min(floor(1000 x / med), INT32_MAX), -1 if E empty
 *   n_eval = |E|, n_flag_rank = #{k in E with bit0}
 *   straggler = n_eval >= min_kernels && score_pm >= 1000 + tau_rank_pm
 * bit3 (degraded pair) = bit0 && !straggler(rank, step).
 * n_flag / n_degraded per (s, k) count bit0 / bit3 over ranks.
 * mean_ns of a present cell = (float)((double)sum / count) (0 when absent).
 */
typedef struct argus_xr_params {
  int32_t min_ranks;   /* >= 1, default 3 */
  int32_t c_min_pair;  /* >= 0, default 8 */
  int32_t min_kernels; /* >= 0, default 8 */
  int32_t k_mad_pm;    /* >= 0, default 5189 (modified z 3.5 = 3.5 / 0.6745 MADs) */
  int32_t ratio_pm;    /* >= 0, default 1250 */
  int32_t alpha_pm;    /* >= 0, default 1500 (Tukey) */
  int32_t tau_rank_pm; /* >= -1000, default 20 */
} argus_xr_params_t;

void argus_xr_default(argus_xr_params_t* p);

typedef struct argus_xr_out {
  /* per (step, kernel), [n_steps][n_kernels] */
  uint32_t* n_present;
  int64_t* med_ns;
  int64_t* mad_ns;
  int64_t* q1_ns;
  int64_t* q3_ns;
  float* xmean_ns;
  uint32_t* n_flag;
  uint32_t* n_degraded;
  /* per cell, [n_ranks][n_steps][n_kernels] */
  float* z;
  float* mean_ns; /* optional (may be NULL) */
  uint8_t* flags;
  /* per (rank, step), [n_ranks][n_steps] */
  int32_t* score_pm;
  uint32_t* n_eval;
  uint32_t* n_flag_rank;
  uint8_t* straggler;
  int32_t* dev_status; /* optional (may be NULL) */
} argus_xr_out_t;

size_t argus_cross_rank_workspace(int32_t n_ranks, int32_t n_steps, int32_t n_kernels);

/* count and sum_ns are argus_summary_t outputs ([n_ranks][n_steps][n_kernels]). */
int argus_cross_rank(const uint32_t* count, const int64_t* sum_ns, int32_t n_ranks, int32_t n_steps,
                     int32_t n_kernels, const argus_xr_params_t* params, const argus_xr_out_t* out, void* workspace,
                     size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------- iter windows
 *
 * Per rank r over y = step_ns[r][0..n_steps) (valid domain 0 <= y < 2^40):
 *  1. window width w = min(W, n_steps); window t covers [t, t+w-1]; it is a
 *     candidate iff 1000 max > theta_pm min.
 *  2. candidate windows that overlap or touch merge into intervals [a, b];
 *     their points get flags bit0.
 *  3. per interval: baseline = lower median of the points outside [a, b]
 *     (of all points when none lie outside); points with 1000 y > beta_pm *
 *     baseline get bit1; the interval's width is its longest run of such
 *     points; eff_width = the largest interval width (0 if none).
 *  4. change point: split t (left [0, t), right [t, S)), both at least
 *     min_seg long, is valid iff sum_left > 0, mean_R / mean_L >= rho_pm /
 *     1000 and both sides have sample (n-1) relative std <= cmax_pm / 1000,
 *     all tested exactly in integers. The valid split with the largest
 *     ratio wins (earliest on ties): cp = t, cp_ratio = (float) ratio, and
 *     steps >= t get bit2; otherwise cp = -1, cp_ratio = 0.
 *  5. cls = (eff_width > 0) | (cp >= 0) << 1: stable 0, jitter 1,
 *     regression 2, both 3. A rank with any y outside the domain gets
 *     cls = 0x80, eff_width 0, cp -1, no flags, and raises ARGUS_DEV_L1_DOMAIN.
 */
typedef struct argus_l1_params {
  int32_t W;        /* >= 1, default 5 */
  int32_t theta_pm; /* >= 0, default 1500 */
  int32_t beta_pm;  /* >= 0, default 1200 */
  int32_t rho_pm;   /* >= 0, default 1300 */
  int32_t cmax_pm;  /* >= 0, default 100 */
  int32_t min_seg;  /* >= 1, default 2 */
} argus_l1_params_t;

void argus_l1_default(argus_l1_params_t* p);

size_t argus_iter_windows_workspace(int32_t n_ranks, int32_t n_steps);

/* cp_ratio and dev_status may be NULL; the other outputs are required. */
int argus_iter_windows(const int64_t* step_ns, int32_t n_ranks, int32_t n_steps, const argus_l1_params_t* params,
                       uint8_t* flags /* [n_ranks][n_steps] */, uint8_t* cls /* [n_ranks] */,
                       int32_t* eff_width /* [n_ranks] */, int32_t* cp /* [n_ranks] */,
                       float* cp_ratio /* [n_ranks] */, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                       void* stream);

/* ---------------------------------------------------------------------- KDE
 *
 * Section 5.2 (Eq. 1): every (rank, step, kernel id) group of valid
 * durations is clustered at the valleys of a Gaussian kernel density
 * estimate over log-duration, and each cluster is summarised as (count, p50,
 * p99). Definition, step by step (every step is exact integer arithmetic
 * except where noted):
 *  1. Grid: x(d) = floor(2^sub_bits * log2 d'), with d' = d truncated to its
 *     24 leading significant bits (exact for d < 2^24) and x(0) = x(1) = 0.
 *     The group's grid is every integer from x(min) to x(max), G points.
 *  2. Bandwidth (Scott's rule as the paper prints it, in grid steps):
 *     var = (n * sum x^2 - (sum x)^2) / (n (n - 1)) evaluated in double from
 *     exact integer sums, h = (1.06 * sqrt(var)) * n^(-1/5) with n^(-1/5) the
 *     double nearest to the real value (decided exactly, no math library),
 *     H = floor(256 h + 0.5); n < 2 gives H = 0. Reported as bw_q8.
 *  3. Density: w(t) = floor(65536 exp(-32768 t^2 / H^2) + 0.5) (double),
 *     f(j) = sum_b c(b) w(|j - b|) over the group's grid histogram c.
 *  4. Valleys (H > 0, G >= 3): each maximal run of equal f strictly below
 *     both neighbouring values, at the middle of the run (rounded down);
 *     a boundary keeps its own grid point in the lower cluster.
 *  5. Cluster-level filter: while the smallest cluster (the lowest one on
 *     ties) has fewer than max(min_count, ceil(frac_pm * n / 1000)) samples,
 *     drop a valley next to it: the only one at either end, else the one
 *     with the larger f (the upper one on ties).
 *  6. Spacing filter: over the boundary list (lowest grid value, valleys,
 *     highest grid value), while two neighbours lie fewer than gap grid
 *     steps apart, take the lowest such pair and drop its valley, or of two
 *     valleys the one with the larger f (the upper one on ties).
 *  7. Cap: while more than ARGUS_KDE_MAXC clusters remain, drop the valley
 *     with the largest f (the upper one on ties).
 *  8. Per cluster, ascending: count; p50 = the lower median and p99 = the
 *     element ceil(0.99 m) (nearest rank) of its m raw durations, sorted.
 * Steps 1-3 approximate Eq. 1: samples are floored onto the grid, the
 * bandwidth comes from the floored values and is rounded to 1/256 step, and
 * the weights are 16-bit integers. Against Eq. 1 evaluated exactly (raw logs,
 * unrounded bandwidth, float64 Gaussian) the tested groups keep the same
 * number of clusters, with at most 6.5e-4 of the samples in another cluster.
 * The only floating-point steps are sqrt and exp in step 2 and 3 (n^(-1/5)
 * is exact by construction); integer outputs follow from them exactly. sqrt
 * and exp are the device's; the weights and bandwidths they give equal those
 * of the host C library on their reachable domain as tested: every weight of
 * every H up to 2^17 and H for 2^22 random (var, n). Thresholds and tie rules
 * are this library's readings: the paper names the filters but gives no
 * values.
 *
 * Inputs: the events (same rules as argus_summarize) and the count, min_ns
 * and max_ns outputs of argus_summarize over those same events. If they do
 * not match, the affected cells report 0 clusters and ARGUS_DEV_KDE_SUMMARY
 * is raised; nothing outside the outputs and the workspace is written.
 * Malformed segments contribute nothing (their summarized counts are 0).
 */
typedef struct argus_kde_params {
  int32_t sub_bits;  /* grid points per octave = 2^sub_bits, 1..6, default 6 */
  int32_t frac_pm;   /* cluster-level filter share in permille, 0..1000, default 50 */
  int32_t min_count; /* cluster-level filter minimum, >= 1, default 3 */
  int32_t gap;       /* spacing filter, grid steps, >= 0, default 48 (0.75 octave at sub_bits 6) */
} argus_kde_params_t;

typedef struct argus_kde_out {
  uint8_t* n_clusters; /* [n_ranks][n_steps][n_kernels]; 0 for empty cells */
  uint32_t* count;     /* [..][ARGUS_KDE_MAXC]; slots past n_clusters are 0 */
  int64_t* p50_ns;     /* [..][ARGUS_KDE_MAXC]; slots past n_clusters are 0 */
  int64_t* p99_ns;     /* [..][ARGUS_KDE_MAXC]; slots past n_clusters are 0 */
  int32_t* bw_q8;      /* optional [..]: H of step 2 */
  int32_t* dev_status; /* optional */
} argus_kde_out_t;

void argus_kde_default(argus_kde_params_t* p);

/* Workspace bytes: 8 per event plus 14 per cell plus 1 per rank-step plus a fixed part. */
size_t argus_kde_workspace(const argus_events_t* ev);

/* ev: as for argus_summarize, n_kernels <= ARGUS_MAX_KDE_KERNELS.
 * sum: count, min_ns and max_ns are read, and n_invalid unless it is NULL: a
 * segment whose n_invalid is 0 holds only valid events, so for id spaces of
 * up to 2,048 kernel ids its stream array is not read (a sixth of the input
 * bytes). sum must be the argus_summarize output of these same events; a
 * summary that does not match them makes the cells concerned report
 * ARGUS_DEV_KDE_SUMMARY. out->count, p50_ns and p99_ns must be 16-byte
 * aligned. The workspace must be 256-byte aligned. */
int argus_kde(const argus_events_t* ev, const argus_summary_t* sum, const argus_kde_params_t* params,
              const argus_kde_out_t* out, void* workspace, size_t workspace_bytes, void* stream);

/* ----------------------------------------------------------------------- W1
 *
 * Section 6.2 (Eq. 2 - 4): the same kernel is compared across ranks through
 * the CDFs reconstructed from each rank's clusters. For every (step s,
 * kernel k), over the ranks whose cell is present (1 <= n_clusters <=
 * ARGUS_KDE_MAXC with cluster counts summing to >= 1; a cell with more
 * clusters, or with total count 0, is malformed: it takes no part and raises
 * ARGUS_DEV_W1_INPUT), n = number of present ranks:
 *  1. Eq. 2: per cluster c, with p50' = max(p50, 1), p99' = max(p99, 1, p50'):
 *     mu_c = ln p50', sigma_c = (ln p99' - mu_c) / 2.326; the rank's CDF is
 *     F(x) = sum_c (count_c / sum count) Phi((ln x - mu_c) / sigma_c), with
 *     Phi(z) = erfc(-z / sqrt 2) / 2, and a unit step at p50' when sigma_c
 *     = 0. All in double, clusters in slot order.
 *  2. Grid: lo = max(1, min over all present clusters of floor(p50'^2 /
 *     p99')), hi = max of min(ceil(p99'^2 / p50'), INT64_MAX) (exact
 *     integers); u_g = ln lo + g (ln hi - ln lo) / (G - 1), x_g = exp(u_g),
 *     g = 0 .. G-1.
 *  3. q_r(g) = min(65535, floor(65536 F_r(x_g))), the CDF in 16-bit fixed
 *     point (F evaluated at u_g directly).
 *  4. Eq. 3 (trapezoid rule), mean over the other ranks: with S_r(g) =
 *     sum_b |q_r(g) - q_b(g)| (exact) and w_g = (x_{min(g+1,G-1)} -
 *     x_{max(g-1,0)}) / 2, score_r = (sum_g w_g S_r(g), added in ascending
 *     g) / (65536 (n - 1)).
 *  5. Eq. 4: q1 = v[(n-1)/4], q3 = v[3(n-1)/4] of the sorted scores v (lower
 *     nearest rank), fence = q3 + alpha_pm (q3 - q1) / 1000, flag = score >
 *     fence; n_flag counts flags.
 * If n < max(min_ranks, 2) the kernel is not evaluated: lo = hi = 0, q1 = q3
 * = fence = 0, n_flag = 0 and its cells get score 0, flag 0. Absent and
 * malformed cells always get score 0, flag 0. Every floating-point step is a
 * double operation in the order written (no contraction); the grid, the
 * 16-bit CDF and the quartile rule are this library's readings: the paper
 * fixes none of them. The logarithm, exponential and erfc are the device
 * library's, so a CDF value that lies within rounding of a multiple of
 * 1/65536 may differ by one unit from another implementation's.
 */
typedef struct argus_w1_params {
  int32_t grid;      /* grid points G, 2 .. ARGUS_MAX_W1_GRID, default 64 */
  int32_t min_ranks; /* >= 1, default 3 */
  int32_t alpha_pm;  /* anomaly coefficient of Eq. 4 in permille, >= 0, default 1500 */
} argus_w1_params_t;

typedef struct argus_w1_out {
  /* per (step, kernel), [n_steps][n_kernels] */
  uint32_t* n_present;
  int64_t* lo_ns;
  int64_t* hi_ns;
  double* q1;
  double* q3;
  double* fence;
  uint32_t* n_flag;
  /* per cell, [n_ranks][n_steps][n_kernels] */
  double* score;
  uint8_t* flag;
  int32_t* dev_status; /* optional (may be NULL) */
} argus_w1_out_t;

void argus_w1_default(argus_w1_params_t* p);

/* Workspace bytes: 2 * n_steps * n_kernels * grid * R' rounded up to a
 * multiple of 256 (the 16-bit CDF values of every rank at every grid point),
 * plus 9 * n_steps * n_kernels * R' (scores and flags on their way to the
 * outputs), R' = n_ranks rounded up to even. */
size_t argus_w1_workspace(int32_t n_ranks, int32_t n_steps, int32_t n_kernels, int32_t grid);

/* clusters: the n_clusters, count, p50_ns and p99_ns outputs of argus_kde
 * ([n_ranks][n_steps][n_kernels] and [..][ARGUS_KDE_MAXC]); count, p50_ns and
 * p99_ns must be 16-byte aligned. n_ranks <= ARGUS_MAX_W1_RANKS, n_steps <=
 * ARGUS_MAX_W1_STEPS. Every output
 * except dev_status is required; the workspace must be 256-byte aligned and
 * not shared by calls that may overlap. */
int argus_w1(const argus_kde_out_t* clusters, int32_t n_ranks, int32_t n_steps, int32_t n_kernels,
             const argus_w1_params_t* params, const argus_w1_out_t* out, void* workspace, size_t workspace_bytes,
             void* stream);

/* ----------------------------------------------------------------------- L2
 *
 * Section 6.1 (parallelism-group-aware routing, Table "routing") and Appendix
 * B (Eq. 5): each event is compared only among the ranks of the parallelism
 * group that its dimension assigns them to. Events are the summaries' kernel
 * ids; the window is one step.
 *
 * Groups: route[e] is the dimension of event e (a value >= n_dims, e.g.
 * 0xFF, means "not compared"); dimension d has up to max_groups groups, group
 * g of d lists members[d][group_off[d][g] .. group_off[d][g+1]) (rank ids).
 * A range that is reversed or leaves [0, n_ranks] is skipped and a member id
 * outside [0, n_ranks) is skipped (ARGUS_DEV_GROUPS_MALFORMED); a rank listed
 * more than once in a dimension counts only at its first listing, the lowest
 * group and then the lowest position (ARGUS_DEV_GROUPS_DUPLICATE).
 *
 * For step s, event e routed to d, group g: x_r = floor((uint64)sum / count)
 * over the listed ranks with count >= 1 and x_r < 2^40 (larger x: left out,
 * ARGUS_DEV_L2_DOMAIN); n of them. With n >= max(min_group, 2), exact
 * integers S = sum x, Q = sum x^2, D = n Q - S^2 (= n (n - 1) sigma^2):
 *   mean = (double)S / n, std = sqrt((double)D / ((double)n (n - 1))),
 *   cv = mean > 0 ? std / mean : 0 (each a double operation);
 *   cls = 0 (balanced) if S = 0 or n D 10^6 < cv_mild_pm^2 (n - 1) S^2,
 *         1 (mild) else if n D 10^6 < cv_severe_pm^2 (n - 1) S^2, else 2;
 *   per member: z = std > 0 ? (float)(((double)x - mean) / std) : 0,
 *   flags bit0 (evaluated) and bit1 (straggler: z > z_pm / 1000, decided as
 *   n x > S and (n x - S)^2 (n - 1) 10^6 > z_pm^2 n D);
 *   n_strag = number of bit1 members.
 * Groups that are not evaluated report n (their present ranks), cls = 0xFF
 * and zeros. Every other cell gets z = 0, flags = 0.
 */
typedef struct argus_l2_params {
  int32_t min_group;    /* >= 2, default 3 */
  int32_t cv_mild_pm;   /* 0 .. 10^6, default 20 (CV 0.02) */
  int32_t cv_severe_pm; /* 0 .. 10^6, default 50 (CV 0.05) */
  int32_t z_pm;         /* 0 .. 10^6, default 3000 (z > 3) */
} argus_l2_params_t;

typedef struct argus_groups {
  const uint8_t* route;     /* [n_events] dimension of each event (device) */
  const int32_t* group_off; /* [n_dims][max_groups + 1] (device) */
  const int32_t* members;   /* [n_dims][n_ranks] (device) */
  int32_t n_dims;           /* 1 .. ARGUS_MAX_L2_DIMS */
  int32_t max_groups;       /* 1 .. 65535, max_groups * n_ranks < 2^32 */
} argus_groups_t;

typedef struct argus_l2_out {
  /* per (step, event, group), [n_steps][n_events][max_groups] */
  uint32_t* n;
  double* mean_ns;
  double* std_ns;
  double* cv;
  uint8_t* cls;
  uint32_t* n_strag;
  /* per cell, [n_ranks][n_steps][n_events] */
  float* z;
  uint8_t* flags;
  int32_t* dev_status; /* optional (may be NULL) */
} argus_l2_out_t;

void argus_l2_default(argus_l2_params_t* p);

/* Workspace bytes: 4 * n_dims * n_ranks (each rank's first listing). */
size_t argus_l2_workspace(int32_t n_ranks, int32_t n_dims);

/* count and sum_ns: argus_summarize outputs ([n_ranks][n_steps][n_events]).
 * n_steps * n_dims <= 65535. The workspace must be 4-byte aligned and not
 * shared by calls that may overlap. */
int argus_l2(const uint32_t* count, const int64_t* sum_ns, int32_t n_ranks, int32_t n_steps, int32_t n_events,
             const argus_groups_t* groups, const argus_l2_params_t* params, const argus_l2_out_t* out,
             void* workspace, size_t workspace_bytes, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* ARGUS_H */
