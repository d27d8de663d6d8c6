/*
 * fbdt.h -- C ABI of libfbdt, a HIP implementation for AMD gfx950 (MI355X)
 * of the fitting and application hot path of FastBDT, the stochastic
 * gradient-boosted decision trees of T. Keck, "FastBDT: A speed-optimized
 * and cache-friendly implementation of stochastic gradient-boosted decision
 * trees for multivariate classification", arXiv:1609.06119.
 *
 * Conventions for every call
 *  - Arrays marked "device" are device pointers that the caller allocates
 *    and owns (e.g. torch tensors on the current HIP device); arrays marked
 *    "host" are ordinary host memory.
 *  - Features are feature-major: element (j, i) of a float array with row
 *    stride ldx is x[j * ldx + i]; binned codes use row stride ldb.
 *    ldb must be a multiple of 16, ldb >= n, and the code buffer must be
 *    16-byte aligned and hold d * ldb bytes.  Bytes of a row beyond n are
 *    read but never influence a result; the binning calls write the first n
 *    bytes of each row only.
 *  - Labels are int8: +1 signal, -1 background (section 1).  Weights are
 *    float32 and finite; NULL means unit weights.  fbdt_fit accepts
 *    negative event weights (section 4.1), as long as each class's total
 *    weight is positive; the single steps take weights >= 0.
 *  - stream is a hipStream_t (NULL = the null stream).  Calls are
 *    stream-ordered; the ones documented as synchronising also wait for it.
 *  - Return value: FBDT_OK (0) or a negative FBDT_E_* code.  On error the
 *    outputs are left untouched where the call checks before it writes (all
 *    argument checks), and fbdt_last_error() describes the failure.
 *  - Calls on distinct models and streams may run concurrently; calls that
 *    fit on the same device serialise on the library's scratch memory.
 *
 * Notation: N events, d features, B bins, D depth, T trees, eta shrinkage,
 * alpha sub-sampling rate.  Node ids are heap-ordered: the root is 1, layer
 * l (0-based) holds nodes [2^l, 2^(l+1)), leaves are [2^D, 2^(D+1)).  A cut
 * (f, c) sends an event to the left child 2n if its bin of feature f is < c
 * and to the right child 2n+1 otherwise (Fig. 1).
 */
#ifndef FBDT_H
#define FBDT_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum fbdt_status {
    FBDT_OK = 0,
    FBDT_E_INVAL = -1,  /* null pointer, size or parameter out of range      */
    FBDT_E_LABEL = -2,  /* a label not in {+1, -1}, or a class with no weight */
    FBDT_E_NAN = -3,    /* NaN among the float features with 256 bins         */
    FBDT_E_WEIGHT = -4, /* a weight not finite                                */
    FBDT_E_SHAPE = -5,  /* too few features for the model                     */
    FBDT_E_DEVICE = -6  /* HIP runtime error or out of device memory          */
};

typedef struct fbdt_model fbdt_model; /* opaque, owned by the library */

/* Hyper-parameters of a fit (sections 1.1-1.4). */
typedef struct {
    int32_t depth;     /* D, number of cut layers, 1..7                        */
    int32_t n_trees;   /* T >= 1, number of boosting steps                     */
    double shrinkage;  /* eta > 0, multiplies every terminal boost weight      */
    double subsample;  /* alpha in (0, 1], per-tree sampling rate              */
    uint64_t seed;     /* seed of the sub-sample generator (SplitMix64)        */
} fbdt_fit_params;

/* A model laid out in plain host arrays (heap order: node k at index k-1). */
typedef struct {
    int32_t n_trees, depth, n_features, n_bins;
    double f0;                  /* initial score: half the weighted log-odds */
    const uint8_t *cut_feature; /* host [T][2^D - 1]                         */
    const uint8_t *cut_bin;     /* host [T][2^D - 1], each in 1..B-1          */
    const double *gain;         /* host [T][2^D - 1] separation gain, or NULL */
    const double *leaf;         /* host [T][2^D], boost weight times eta      */
    const float *boundaries;    /* host [d][B - 1] bin boundaries, or NULL    */
    /* host [T][2^D - 1] boost weight times eta of every inner node, or NULL.
     * Present when the model handles missing values (section 4.2): with at
     * most 255 bins, bin code 255 marks a missing value, and an event whose
     * code (apply) or value (apply_float: NaN) of a node's cut feature is
     * missing stops at that node and takes its weight. */
    const double *inner;
} fbdt_model_view;

/*
 * Equal-frequency binning of a training sample (section 2.2, Fig. 3).
 * For each feature j, with s the ascending sort of the m non-NaN values of
 * x[j][0..n), boundary k (k = 1..B-1) is s[floor(k m / B)] (+inf when m = 0)
 * and a value goes to bin #{k : boundary_k <= value}.  Tied values share a
 * bin; repeated boundaries leave empty bins.  NaN values are missing
 * (section 4.2): with n_bins <= 255 they take the reserved code 255, with
 * 256 bins they are an error (FBDT_E_NAN).  x: device float32 [d][ldx];
 * boundaries: host float32 [d][B-1] (output); xb: device uint8 [d][ldb]
 * (output; only the first n bytes of each row are written).  1 <= d <= 255,
 * 2 <= n_bins <= 256, n >= 1.  The sort runs on the device (one radix sort
 * per batch of features, scratch held by the library); the call
 * synchronises the stream.
 */
int fbdt_bin(const float *x, int64_t n, int32_t d, int64_t ldx, int32_t n_bins,
             float *boundaries, uint8_t *xb, int64_t ldb, void *stream);

/*
 * Bin fresh events with the boundaries of a training sample (section 2.2).
 * Same layouts as fbdt_bin; boundaries is host input.  A NaN value takes
 * code 255 with n_bins <= 255 and is an error (FBDT_E_NAN) with 256 bins;
 * the stream is synchronised to report it.
 */
int fbdt_bin_transform(const float *x, int64_t n, int32_t d, int64_t ldx, int32_t n_bins,
                       const float *boundaries, uint8_t *xb, int64_t ldb, void *stream);

/*
 * Fit T trees of depth D by stochastic gradient boosting (sections 1.1-1.4,
 * 2.1) on binned features: two-class LK_TreeBoost with a SplitMix64
 * Bernoulli sub-sample per tree, per-layer signal/background histograms of
 * all nodes and features in one pass, cumulative histograms, weighted Gini
 * separation gain, lowest-(feature, bin) argmax (gains that agree in all
 * but the last 16 of their 52 mantissa bits count as tied), and Newton-step
 * terminal weights.  xb: device uint8 [d][ldb]; y: device int8 [n]; w: device
 * float32 [n] or NULL (event weights, any sign; each class's total must be
 * positive, else FBDT_E_LABEL); score_out: optional device float64 [n] that receives
 * the final score F of every event.  Codes must be < n_bins, except that
 * with n_bins <= 255 code 255 marks a missing value (section 4.2): it stays
 * out of its feature's histograms, an event stops at the node that cuts on
 * a feature it misses, and every node, inner or leaf, gets a boost weight
 * over the sampled events that reached it (the model's inner weights).
 * Other codes >= n_bins give FBDT_E_INVAL.
 * *out receives a new model (free with fbdt_model_free).  Synchronises the
 * stream before returning.
 */
int fbdt_fit(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb, int32_t n_bins,
             const int8_t *y, const float *w, const fbdt_fit_params *params,
             fbdt_model **out, double *score_out, void *stream);

/*
 * Score events (Fig. 1, section 1.3): F = f0 + sum over trees of the leaf
 * reached, accumulated in float64 in tree order; prob = 1 / (1 + exp(-2F))
 * rounded to float32.  A model with inner weights (missing values) stops an
 * event at the node whose cut feature has code 255 and adds that node's
 * weight.  xb: device uint8 [d][ldb] with d >= the model's feature count
 * (else FBDT_E_SHAPE); prob: device float32 [n] (output); score: optional
 * device float64 [n] (output).  Stream-ordered, except that the first call
 * for a model on a device (or launch shape) uploads the model's arrays
 * with a synchronous copy and allocates their device copy, which the model
 * owns until fbdt_model_free.
 */
int fbdt_apply(const fbdt_model *m, const uint8_t *xb, int64_t n, int32_t d, int64_t ldb,
               float *prob, double *score, void *stream);

/*
 * Score float32 events without binning them (section 2.2, the inverse of the
 * bin transform): the cut "bin >= c" of feature j is the test
 * x >= boundaries[j][c - 1], which holds exactly when the value's bin (the
 * number of boundaries at or below it) is >= c, so for events without NaN
 * values the result equals fbdt_apply on fbdt_bin_transform's codes bit for
 * bit (NaN: see below; fbdt_bin_transform gives NaN code 255, which in a
 * model without inner weights goes right at every cut).  The model needs its
 * boundaries (fbdt_model_set_boundaries or fbdt_model_import), else
 * FBDT_E_INVAL.  x: device float32 [d][ldx], ldx >= n, d >= the model's
 * feature count (else FBDT_E_SHAPE).  A NaN value stops the event at the
 * node that cuts on it when the model has inner weights (as code 255 does
 * in fbdt_apply); in other models it fails every test and takes the left
 * branch, as code 0 would.  prob, score as for fbdt_apply.  Stream-ordered.
 */
int fbdt_apply_float(const fbdt_model *m, const float *x, int64_t n, int32_t d, int64_t ldx,
                     float *prob, double *score, void *stream);

/*
 * Global feature importance (section 4.3): the separation gains of all
 * nodes of all trees summed per cut feature, in tree order then heap order.
 * importance: host float64 [the model's feature count] (output).
 */
int fbdt_feature_importance(const fbdt_model *m, double *importance);

/*
 * Importance of every feature for every event (section 4.3): the gains of
 * the nodes on the event's path through the trees summed per cut feature,
 * tree by tree in float64; with missing values a path ends at the node
 * whose cut feature the event misses, without that node's gain.  xb: device
 * uint8 [d][ldb] (as fbdt_apply);
 * importance: device float64 [d][ldi] (output, ldi >= n; rows of features
 * beyond the model's are zero).  Stream-ordered.
 */
int fbdt_event_importance(const fbdt_model *m, const uint8_t *xb, int64_t n, int32_t d,
                          int64_t ldb, double *importance, int64_t ldi, void *stream);

/* Borrowed host view of a model, valid until fbdt_model_free: the forest of
 * Fig. 1 (cuts in heap order, terminal boost weights of section 1.3), f0,
 * the separation gains (section 4.3) and the bin boundaries (section 2.2). */
int fbdt_model_export(const fbdt_model *m, fbdt_model_view *view);

/* New model from host arrays (copied), in the layout of fbdt_model_export;
 * gain and boundaries may be NULL.  Cut features must be < n_features and
 * cut bins in 1..n_bins-1, else FBDT_E_INVAL.  Boundaries, if given, must
 * hold no NaN and ascend (non-strictly) per feature, else FBDT_E_INVAL. */
int fbdt_model_import(const fbdt_model_view *view, fbdt_model **out);

/*
 * Attach the training sample's bin boundaries (host float32 [d][B - 1], as
 * fbdt_bin returns them; copied) to a model, for fbdt_apply_float.  They
 * must hold no NaN and ascend per feature, else FBDT_E_INVAL.  Not to be
 * called while the model is applied on another thread.
 */
int fbdt_model_set_boundaries(fbdt_model *m, const float *boundaries);

/* Frees a model made by fbdt_fit or fbdt_model_import and its device
 * copies; NULL is ignored.  Not to be called while the model is in use. */
void fbdt_model_free(fbdt_model *m);

/* Message of the last failed call on this thread ("" if none): the argument
 * or device condition behind the FBDT_E_* code the call returned.  Owned by
 * the library, valid until the thread's next failing call. */
const char *fbdt_last_error(void);

/* ---- The steps of one boosting iteration, callable one at a time ------- */
/* With n_bins <= 255, fbdt_histogram leaves code 255 (a missing value) out
 * of its sums; fbdt_route and fbdt_leaf_values know no stops at missing
 * values, which fbdt_fit handles itself. */

/*
 * Re-weighting of one tree (sections 1.3, 1.4): for every event,
 * y~ = 2y / (1 + exp(2 y F)); sampled iff the (tree * n + i)-th SplitMix64
 * output of seed, top 53 bits over 2^53, is < alpha; w_out = |fl32(v |y~|)|
 * if sampled, else 0, carrying the class in its sign (+ signal,
 * - background).  y, v (NULL = unit), F: device [n]; w_out: device float32
 * [n].  Stream-ordered.
 */
int fbdt_tree_weights(const int8_t *y, const float *v, const double *F, int64_t n,
                      uint64_t seed, int32_t tree, double alpha, float *w_out, void *stream);

/*
 * Signal/background histograms of every node and feature of one layer
 * (sections 1.1, 2.1): hist[k][j][b][c] = sum of |w_i| over events with
 * node_i = 2^layer + k, bin b in feature j, class c (0 = signal, w > 0;
 * 1 = background, w < 0); events with w = 0 are skipped.  node: device
 * uint8 [n] heap ids of the layer; w: device float32 [n] as produced by
 * fbdt_tree_weights; hist: device float64 [2^layer][d][B][2] (output,
 * overwritten).  0 <= layer <= 6.  Stream-ordered.
 */
int fbdt_histogram(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb, int32_t n_bins,
                   const uint8_t *node, const float *w, int32_t layer, double *hist,
                   void *stream);

/*
 * Cumulative histograms, separation gains and best cut of every node of a
 * layer (section 1.1).  For node k and feature j with cumulative sums S(c),
 * B(c) of the bins below c and totals S_T, B_T:
 *   gain(c) = (G(S_T, B_T) - G(S(c), B(c))) - G(S_T - S(c), B_T - B(c)),
 *   G(s, b) = s b / (s + b), 0 when s + b = 0, for c = 1..B-1;
 * the cut is the highest gain, ties to the lowest feature, then bin.
 * hist: device float64 [n_nodes][d][B][2]; cut_feature, cut_bin: device
 * uint8 [n_nodes]; gain: device float64 [n_nodes].  Stream-ordered.
 */
int fbdt_best_cuts(const double *hist, int32_t n_nodes, int32_t d, int32_t n_bins,
                   uint8_t *cut_feature, uint8_t *cut_bin, double *gain, void *stream);

/*
 * fbdt_best_cuts for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same result, bit for bit, from the same kernels, but the candidate
 * cuts live in a fixed device array of the library (192 KiB per device, held
 * until the process ends) instead of its allocated scratch.  The call makes
 * no allocation and does not synchronise (stream-ordered).  Limit: n_nodes *
 * d <= 16384, which n_nodes <= 64 and d <= 255 always meet.  Every call on a
 * device shares that device's array: calls that overlap on one device (other
 * streams, other threads) race and must be ordered by the caller.
 */
int fbdt_best_cuts_noalloc(const double *hist, int32_t n_nodes, int32_t d, int32_t n_bins,
                           uint8_t *cut_feature, uint8_t *cut_bin, double *gain, void *stream);

/*
 * Route every event one layer down (section 1.1): node <- 2 node +
 * [xb[f][i] >= c] with (f, c) the cut of its node.  node: device uint8 [n],
 * updated in place (ids of `layer` on entry); cut_feature, cut_bin: device
 * uint8 [2^layer].  Stream-ordered.
 */
int fbdt_route(const uint8_t *xb, int64_t n, int32_t d, int64_t ldb, uint8_t *node,
               const uint8_t *cut_feature, const uint8_t *cut_bin, int32_t layer,
               void *stream);

/*
 * Terminal boost weights of one tree (section 1.3, Friedman's Newton step):
 * leaf[j] = eta * sum(v y~) / sum(v |y~| (2 - |y~|)) over the sampled
 * events of leaf j (0 if the denominator is 0), with y~ and the sample as
 * in fbdt_tree_weights.  node: device uint8 [n] leaf heap ids (2^D..);
 * leaf: device float64 [2^D] (output).  Stream-ordered.
 */
int fbdt_leaf_values(const uint8_t *node, const int8_t *y, const float *v, const double *F,
                     int64_t n, int32_t depth, uint64_t seed, int32_t tree, double alpha,
                     double eta, double *leaf, void *stream);

/* ---- Measurement and tuning -------------------------------------------- */

enum fbdt_kernel_kind {
    FBDT_K_HISTOGRAM = 0, /* per-layer histogram pass (routing fused up to 4  */
                          /* parents)                                         */
    FBDT_K_BEST_CUTS = 1, /* CPH scan, gain and argmax of one layer          */
    FBDT_K_TREE_PREP = 2, /* score update and re-weighting of one tree       */
    FBDT_K_LEAF = 3,      /* last routing and terminal boost weights          */
    FBDT_K_APPLY = 4,     /* forest traversal                                */
    FBDT_K_ENCODE = 5,    /* float -> bin code                                */
    FBDT_K_ROUTE = 6,     /* routing of a layer as a pass of its own (layers  */
                          /* with more than 4 parents; fbdt_route)            */
    FBDT_K_REFERENCE = 7, /* fbdt_reference_pass                              */
    FBDT_K_COUNT = 8
};

/*
 * Kernel timing with HIP events recorded on the launching stream around
 * every launch of the selected kinds (bit k of `kinds` selects kind k;
 * 0 turns timing off, the default).  The call resets the tallies.
 * fbdt_timing_read waits for the recorded events and returns
 * the number of launches of a kind, their summed duration in milliseconds
 * and the summed algorithmic bytes those launches move (histogram: codes,
 * node ids, weights, routing and the histogram written; route: parent id,
 * one code and the new id per event; 0 where not counted).
 */
int fbdt_timing_enable(int32_t kinds);
int fbdt_timing_read(int32_t kind, int64_t *launches, double *total_ms, double *bytes);

/*
 * Launch-shape overrides for sweeps; value 0 restores the default.
 * Names: "hist_features_per_group" (1, 2, 4, 5 or 8), "hist_event_chunks",
 * "hist_threads" (a multiple of 64, at most 1024), "hist_copies" (1, 2 or 4
 * LDS copies of a workgroup's histograms), "apply_threads".
 * "fit_graphs" (default 1): fbdt_fit records the kernel launches of its
 * boosting loop as a HIP graph on first use of an argument set (device,
 * buffer addresses, sizes, parameters, launch shapes) and replays it on later
 * calls with the same set; up to 4 graphs per device are kept, and growing the
 * device workspace drops them.  0 launches every kernel one by one.  Graphs
 * are not used while any fit kernel kind is being timed.
 * "fail_alloc" (default 0, for tests of the error path): the next `value`
 * device allocations the library would make (its scratch, a model's device
 * copy) fail instead, and the calls that needed them return FBDT_E_DEVICE;
 * a positive value first releases the scratch the library holds (waiting
 * for the devices to finish with it), so the next call that needs scratch
 * allocates.
 * "hist_timeline" (default 0): 1 makes fbdt_fit record the phase timeline
 * of every histogram launch (see fbdt_hist_timeline); fits then launch
 * kernel by kernel and stream every layer (no event lists).
 * "hist_lists" (default 0: fits with n * (depth - 2) >= 10,000,000): how fbdt_fit
 * builds the histograms of the layers below the root (sections 1.1, 2.1).
 * 1 streams every event through every layer's pass; 2 has each layer's
 * routing pass append the sampled events of one child of every parent (the
 * one with less weight in the parent's histograms) to per-parent lists,
 * with missing values (section 4.2) also the events that stop at the parent
 * to a list of their own, and histograms the lists, the codes read from an
 * event-major copy of the code matrix (n * round_up(d, 16) bytes of device
 * workspace, plus 8 bytes per event for the lists, 16 with missing values);
 * the other child is the parent minus the lists.  Fits need n < 2^31 for it.  Both give the same model bit
 * for bit, except for the rounding of sums of weights below the
 * fixed-point grid.  "list_features_per_group" (4, 8, 12, 20, 28, 36 or
 * 40), "list_parts" (workgroups per feature group, at most 4096) and
 * "list_copies" (1, 2 or 4) override the list pass's launch shape.
 * Returns FBDT_E_INVAL for an unknown name.
 */
int fbdt_set_option(const char *name, int64_t value);

/*
 * Phase timeline of the histogram launches of the last fbdt_fit made while
 * option "hist_timeline" was 1 (measurement of the layer pass of sections
 * 1.1 and 2.1).  Launch k = tree * D + layer ran blocks[k] workgroups;
 * workgroup b of it wrote stamps[(k * max_blocks + b) * 5 + p], the value
 * of the device's constant-rate clock (rate_khz ticks per millisecond) at
 * phase p: 0 entry, 1 the parents' cuts in LDS, 2 first step of events
 * added (wavefront 0), 3 every add done, 4 partial rows written (wavefront
 * 0).  A row is 0 for workgroups beyond the launch's work and phase 2 is 0
 * for a workgroup without events.  The arrays belong to the library and
 * stay valid until the next such fit (or the end of the process); launches
 * = 0 if there was none.
 */
int fbdt_hist_timeline(int64_t *launches, int32_t *max_blocks, const int32_t **blocks,
                       const uint64_t **stamps, int64_t *rate_khz);

/*
 * Reference passes for the histogram pass's roofline (measurement of the
 * layer pass of sections 1.1 and 2.1): launched with the grid, workgroup
 * size and dynamic LDS that fbdt_fit uses for `layer` of n events x d
 * features at n_bins, kind 0 runs workgroups that return at once (launch
 * cost) and kind 1 workgroups that read what the pass reads (the weights,
 * the node ids if node is not NULL, and the codes of their features over
 * their event chunk) and write nothing.  xb as for fbdt_histogram; w
 * (float32) and node (uint8, or NULL) on the device, holding round_up(n, 8)
 * elements, 16-byte aligned.  Timed as FBDT_K_REFERENCE with the bytes read.
 * Stream-ordered.
 */
int fbdt_reference_pass(int32_t kind, const uint8_t *xb, int64_t n, int32_t d, int64_t ldb,
                        int32_t n_bins, int32_t layer, const uint8_t *node, const float *w,
                        void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FBDT_H */
