// Internal launch interface between the C ABI (capi.hip) and the kernels
// (kernels.hip).  Nothing here is exported from libfbdt.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace fbdt {

// Bits of the device-side error word that kernels raise.
enum : int {
    kErrLabel = 1,     // label not in {+1, -1}
    kErrWeight = 2,    // weight not finite
    kErrNan = 4,       // NaN feature value
    kErrBin = 8,       // bin code >= n_bins met by a histogram pass
    kErrRoute = 16,    // cut or node id out of range met while routing
    kErrClass = 32,    // a class has no positive total weight
    kNegWeights = 64,  // (not an error) some event weight is negative
    kHasMissing = 128, // (not an error) some bin code is the missing code
};

// Missing values (section 4.2): with at most kMissingCode bins a NaN value
// takes the bin code kMissingCode; it stays out of the feature's histograms,
// and an event whose code of a node's cut feature is kMissingCode stops at
// that node (its terminal node, whose boost weight it takes).
constexpr int kMissingCode = 255;

// Launch shape of one histogram pass.
struct HistShape {
    int features_per_group;   // features whose histograms one workgroup keeps in LDS
    int feature_groups;       // ceil(d / features_per_group)
    int nodes_per_group;      // nodes whose histograms one workgroup keeps in LDS
    int node_groups;          // ceil(2^layer / nodes_per_group)
    int chunks;               // event chunks, each merged once per layer: the same number
                              // in each XCD's event range (a multiple of kXcds)
    int64_t chunk_events;     // events per chunk (a multiple of kHistE = 8)
    int64_t xcd_events;       // events of an XCD's range, xcd_range(n)
    int threads;              // threads per workgroup
    int blocks;               // grid size (chunks * groups, rounded up to the XCD count)
    int copies;               // LDS copies of the workgroup's histograms (1, 2 or 4):
                              // lane l adds into copy l % copies
    int copy_stride;          // bytes between copies (the histograms plus a bank shift)
    size_t lds_bytes;         // dynamic LDS per workgroup
    bool sibling;             // routed pass below the root histograms the left child of
                              // each parent only (right = parent - left)
    bool prefix;              // partial rows written as inclusive prefix sums over bins
                              // (the fit's passes, read by the cut scan); the planner
                              // leaves it false (plain rows, for merge_partials)
};

// Launch-shape overrides of the histogram pass (0 = the planner's choice).
struct HistOverrides {
    int fpg = 0, chunks = 0, threads = 0, copies = 0;
};

// Device-side scratch of one fit.
struct FitBuffers {
    double *F;            // [npad] score
    float *w;             // [npad] signed re-weighted sample
    double *yts;          // [npad] y~ of the sampled events, 0 for the others
    float *v;             // [npad] caller's event weights, padded (null: unit weights)
    uint8_t *node[2];     // [npad] node ids, double-buffered across layers
    uint64_t *partial;    // fixed-point histogram partials [chunks][histogrammed nodes][d][B][2]
    uint64_t *hfull[2];   // summed fixed-point histograms of every node of a layer
                          // [nodes][d][B][2], by layer parity (the next layer's parents)
    double *small[2];     // float64 histograms of the weights below the fixed-point grid,
                          // [nodes][d][B][2], by the parity of tree * D + layer
    uint32_t *sany;       // [2] non-zero once a list route pass added to small[p] (cleared
                          // with it)
    unsigned long long *keys;   // [2][kKeyWords] best-cut keys of a layer's nodes, by the
                                // parity of tree * D + layer
    double *cand_gain;    // [max nodes][d * slices] best gain of every (node, feature, slice)
    int *cand_cut;        // [max nodes][d * slices] and its bin
    double *leaf_partial;   // [leaf blocks][2^D][2]
    double *class_partial;  // [validate blocks][3]: signal, background, sum of |v|
    uint8_t *vsign;         // [npad] 1 = negative event weight (fits with negative weights)
    double *f0;             // [2]: initial score, sum of |v| (bounds every histogram sum)
    int *err;               // [1]
    uint8_t *cut_feature;   // [T][2^D - 1]
    uint8_t *cut_bin;       // [T][2^D - 1]
    double *gain;           // [T][2^D - 1]
    double *leaf;           // [T][2^D]
};

constexpr int kXcds = 8;            // gfx950: 8 XCDs, workgroups dispatched round-robin
constexpr int kXcdQuantum = 64;     // XCD event ranges are whole multiples of this

// Every per-event pass of a fit gives the events [x R, min(n, (x + 1) R)),
// R = xcd_range(n), to workgroups on XCD x (workgroup b runs on XCD b % 8),
// so that the per-event arrays one pass writes stay in that XCD's L2 for the
// next pass: R = ceil(n / 8) rounded up to kXcdQuantum.
int64_t xcd_range(int64_t n);
constexpr int kValidateBlocks = 256;
// LDS kept aside for a kernel's static shared arrays when sizing its
// dynamic LDS (the histogram kernel's cut table takes 128 bytes)
constexpr size_t kHistStaticLdsReserve = 1024;
// bytes between LDS copies of the histograms beyond their size: a shift of
// 16 four-byte banks, so that copy c of a counter sits 16 c banks away
constexpr size_t kHistCopyShift = 64;
// chunk length (events per workgroup) from which the planner uses copies
constexpr int64_t kHistCopiesMinEvents = 131072;
// features per histogram workgroup the kernels are built for (a workgroup
// holds the codes of all of them in registers per step)
constexpr int kHistFpgSizes[] = {1, 2, 4, 5, 8};
constexpr int kHistFMax = 8;
bool hist_fpg_supported(int f);

// Sets the per-kernel attributes the launchers rely on (dynamic LDS above
// 64 KiB) for the current device; called once per device before any launch,
// so that a launch sequence holds nothing but kernel launches.
hipError_t prepare_kernels(size_t max_lds);

hipError_t launch_fill_u32(void *p, uint32_t value, size_t count, hipStream_t s);

hipError_t launch_validate(const int8_t *y, const float *v, int64_t n, double *class_partial,
                           int *err, hipStream_t s);
// err |= flag if any of the first n codes of a row equals `code`.
hipError_t launch_find_code(const uint8_t *xb, int64_t ldb, int64_t n, int d, uint8_t code,
                            int flag, int *err, hipStream_t s);
hipError_t launch_initial_score(const double *class_partial, double *f0, int *err,
                                hipStream_t s);

// Deepest tree whose boost weights tree_prep sums from the leaf-pass
// partials itself (2^depth leaves, two sums each, per workgroup partial).
constexpr int kFusedLeafDepth = 4;

// Score update of the previous tree (if any) and re-weighting of tree `tree`.
//  leaf_partial != null (depth <= kFusedLeafDepth): the previous tree's boost
//    weights are summed from the leaf-pass partials (lblocks of them) and
//    eta; leaf_rec (optional) receives them;
//  else leaf_prev != null: the previous tree's boost weights;
//  either way F += weight[leaf_node - 2^depth]; else if f0 != null: F = *f0.
//  w may be null (score update only); yts (optional) receives y~ of the
//  sampled events and 0 for the others; score_out (optional) receives F.
hipError_t launch_tree_prep(const int8_t *y, const float *v, double *F, const double *f0,
                            const uint8_t *leaf_node, const double *leaf_prev,
                            const double *leaf_partial, int lblocks, double eta, double *leaf_rec,
                            int depth, bool missing, int64_t n, uint64_t seed, int tree,
                            double alpha, float *w, double *yts, double *score_out, int cu_count,
                            hipStream_t s);

// ov: launch-shape overrides (0 = the planner's choice).  sibling: the
// routed fit pass, which for layer >= 1 histograms one child per parent.
HistShape plan_histogram(int64_t n, int d, int n_bins, int layer, bool sibling, int cu_count,
                         size_t max_lds, const HistOverrides &ov);

// Best-cut keys of a layer's nodes: the cut scan takes the maximum of every
// candidate's 64-bit key (gain order, then lowest feature and bin) into
// keys[(node * kXcds + x) * kKeyStride], a slot per node and XCD x of the
// candidate's workgroup (one 128-byte line each, so that the atomics of a
// node spread over 8 lines); the node's key is the maximum of its slots; 0 =
// no candidate.  Two buffers of kKeyNodes nodes, used by alternate layers.
constexpr int kKeyStride = 16;
constexpr int kKeyNodes = 64;
constexpr size_t kKeyWords = (size_t)kKeyNodes * kXcds * kKeyStride;   // per buffer

// The cuts a routed pass takes for the parents of its layer: their best-cut
// keys, and the candidates (gain of the best cut of each (node, feature,
// slice)) whose gain rec_g receives; rec_* (optional) receive the cuts for
// the model (written by workgroup 0).
struct ParentCuts {
    const double *cand_gain = nullptr;   // [nodes][d * slices]
    const unsigned long long *keys = nullptr;
    int slices = 1;
    uint8_t *rec_f = nullptr;
    uint8_t *rec_c = nullptr;
    double *rec_g = nullptr;
};

// Fixed-point scale of the histogram sums: a weight w >= 2^(23 - scale) is
// an exact multiple of 2^-scale and is added as the integer w * 2^scale;
// smaller positive weights go to a float64 side histogram.  The scale is
// chosen so that no bin total can reach 2^63: total_weight_bound * 2^scale
// < 2^62.
int histogram_scale(double total_weight_bound);

// Histogram pass.  routed = true: node_in holds the ids of layer-1 (null for
// layer <= 1, all events at the root), the pass routes them with the cuts of
// layer-1 (from pc) and (first feature group only) writes the layer's ids to
// node_out; for layer >= 1 it histograms only the left child of every
// parent (the right child is the parent minus the left child, formed by
// best_cuts): partial: [chunks][2^(layer-1)][d][B][2], indexed by parent.
// routed = false: node_in holds the ids of the layer itself; partial:
// [chunks][2^layer][d][B][2], or with hs.sibling (layer >= 1, ids written by
// launch_route_layer) [chunks][2^(layer-1)][d][B][2] of the left children
// only, indexed by parent.  Ids below the layer (events stopped earlier at
// a missing value) count nowhere.
// small: [2^layer][d][B][2] float64 sums of the weights below the grid, for
// every node of the layer (accumulated into, not cleared).
// Every step reads kHistE = 8 whole events: w and node_in must hold
// round_up(n, 8) elements, with weight 0 beyond n (those events count
// nowhere), code rows ldb >= round_up(n, 8) bytes, and node_out room for
// round_up(n, 8) ids (the padded events are routed too).
// vsign (or null): [round_up(n, 8)] bytes, 1 where the
// event's weight is negative; w then holds |w| with the class in the sign
// bit and the pass adds -|w| for those events (two's complement fixed point).
// tl (optional, measurement): kTimelineStamps clock values per workgroup of
// the launch (hs.blocks rows), see fbdt_hist_timeline.
constexpr int kTimelineStamps = 8;
hipError_t launch_histogram(const HistShape &hs, const uint8_t *xb, int64_t ldb, int64_t n,
                            int d, int n_bins, const uint8_t *node_in, uint8_t *node_out,
                            const float *w, const uint8_t *vsign, const ParentCuts &pc,
                            int layer, bool routed, int scale, uint64_t *partial, double *small,
                            int *err, hipStream_t s, unsigned long long *tl = nullptr);

// Reference passes of the histogram pass (measurement): the pass's grid,
// workgroup size and LDS for shape hs; kind 0 returns at once, kind 1 reads
// the weights, node ids (node may be null) and its features' codes.
hipError_t launch_hist_reference(int kind, const HistShape &hs, const uint8_t *xb, int64_t ldb,
                                 int64_t n, int d, const uint8_t *node, const float *w,
                                 uint32_t *sink, hipStream_t s);

// vs[i] = 1 where v[i] < 0 (i < n), else 0, for i < npad.
hipError_t launch_sign_bytes(const float *v, int64_t n, int64_t npad, uint8_t *vs, hipStream_t s);

// hist[i] = (sum over chunks of partial[chunk][i]) * 2^-scale + small[i].
hipError_t launch_merge_partials(const uint64_t *partial, int chunks, size_t count, int scale,
                                 const double *small, double *out, hipStream_t s);

// Sum of |w| over n weights into *out (fixed order).
hipError_t launch_abs_sum(const float *w, int64_t n, double *block_partial, double *out,
                          hipStream_t s);

// Slices of the candidate cuts of one (node, feature) row: ceil((B-1)/31).
int cut_slices(int n_bins);

// Best cut of every (node, feature) of a float64 histogram hist
// [n_nodes][d][B][2] into cand_gain/cand_cut [n_nodes][d] (one slice per
// feature).
hipError_t launch_best_cuts_f64(const double *hist, int n_nodes, int d, int n_bins,
                                double *cand_gain, int *cand_cut, hipStream_t s);

// Best cuts of a layer in the fit from the prefix-summed fixed-point chunk
// partials of the histogram pass (hnodes slots, chunks partials) plus the
// float64 side histogram `small` of the layer, into cand_gain/cand_cut
// [layer nodes][d * cut_slices(B)].  mode kCutSibling (layers below the
// root): slot k holds the left child of parent k and hparent [parents][d][B]
// [2] the parents' summed prefix rows; the right child is parent - left.
// kCutStopped: slot 2k the left child, slot 2k + 1 the events that stopped
// at parent k; the right child is parent - left - stopped.  hout (optional)
// receives the summed prefix rows of every node of the layer.  Clears
// small_next[0, small_next_count) (the next layer's side histogram) and
// *sany_next (if given).  sany (list layers, or null): the side histogram
// is read only if *sany is non-zero (the route pass added to it).
// lchunks (list passes): the partials of slot k are the rows [x_k, x_k +
// (y_k & 0x7fffffff)) of [*][d][B][2], and bit 31 of y_k tells that a
// child slot holds the right child (the left is then the one formed).
// clear_words (optional): clear_count words zeroed on the way.  keys
// (optional): each node's best-cut key slots (kKeyWords, zero on entry), the
// maximum of its candidates' keys; keys_next (optional): the next layer's,
// cleared on the way.
enum CutMode : int {
    kCutPlain = 0,     // slot k holds node k
    kCutSibling = 1,   // slot k holds one child of parent k, the other is parent - child
    kCutStopped = 2,   // slot 2k holds one child of parent k, slot 2k + 1 the events that
                       // stopped at k; the other child is parent - child - stopped
};
hipError_t launch_cut_scan(const uint64_t *partial, int chunks, int scale, const double *small,
                           const uint32_t *sany, double *small_next, uint32_t *sany_next,
                           size_t small_next_count, int hnodes, int d,
                           int n_bins, int mode, double *cand_gain, int *cand_cut,
                           const uint64_t *hparent, uint64_t *hout, hipStream_t s,
                           const uint2 *lchunks = nullptr, uint32_t *clear_words = nullptr,
                           int clear_count = 0, unsigned long long *keys = nullptr,
                           unsigned long long *keys_next = nullptr);

// Best cut of each node over its candidates (d features x slices entries).
hipError_t launch_select_cuts(const double *cand_gain, const int *cand_cut, int n_nodes, int d,
                              int slices, uint8_t *out_f, uint8_t *out_c, double *out_g,
                              hipStream_t s);

// Last routing (routed = true, from layer depth-1 to the leaves with the
// cuts from pc) or none (node_in already holds leaf ids), then the per-block
// partial sums of the terminal boost weights from yts (y~ of the sampled
// events, 0 for the others); launch_leaf_finalize adds the partials and
// writes eta * num / den per leaf.  node_in, v (or null: unit weights) and
// yts hold round_up(n, 8) elements with yts = 0 beyond n; node_out receives
// round_up(n, 8) ids.
// missing (section 4.2): the terminal nodes are every node of the tree, in
// heap order (slot k - 1 = node k), and an event whose code of its node's
// cut feature is kMissingCode stays at that node; launch_leaf_finalize then
// writes the boost weight of every node, an inner node's over all the
// sampled events that reached it.  The leaf pass of depth 7 with missing
// values needs more LDS than a CU has (hipErrorInvalidValue).
int leaf_blocks(int64_t n, int depth, bool missing, int cu_count);
size_t leaf_lds_bytes(int depth, bool missing);
constexpr size_t kLeafMaxLds = 136 * 1024;
hipError_t launch_leaf(const uint8_t *xb, int64_t ldb, int64_t n, int d, const uint8_t *node_in,
                       uint8_t *node_out, const ParentCuts &pc, int depth, bool missing,
                       bool routed, const float *v, const double *yts, int blocks,
                       double *leaf_partial, int *err, hipStream_t s);
hipError_t launch_leaf_finalize(const double *leaf_partial, int blocks, int depth, bool missing,
                                double eta, double *leaf_out, hipStream_t s);

hipError_t launch_route(const uint8_t *xb, int64_t ldb, int64_t n, int d, uint8_t *node,
                        const uint8_t *cut_f, const uint8_t *cut_c, int layer, int *err,
                        hipStream_t s);

// The histogram pass routes the events itself while the layer has at most
// this many parents (it loads the parents' cut-feature rows with the codes);
// deeper layers are routed by launch_route_layer first.
constexpr int kRoutedMaxParents = 4;

// Routing of layer `layer` (>= 1) on its own: the parents' cuts from their
// best-cut keys in pc (recorded in the model through pc.rec_*), then
// node_out[i] = 2 node_in[i] + [code >= cut] for every event up to
// round_up(n, 8); with miss (n_bins <= kMissingCode) an event whose code of
// the cut feature is kMissingCode, or whose id lies below the parents'
// layer, keeps its id.
hipError_t launch_route_layer(const uint8_t *xb, int64_t ldb, int64_t n, int d,
                              const uint8_t *node_in, uint8_t *node_out, const ParentCuts &pc,
                              int layer, bool miss, int *err, int cu_count, hipStream_t s);

// Event lists of the histogrammed nodes ("slots": the left child of every
// parent, or with missing values every node of the layer), for layers 1 ..
// depth - 1 of large fits.  launch_route_list routes a layer (as
// launch_route_layer) and appends each sampled event that the layer's
// histograms count and whose weight is on the fixed-point grid to its
// slot's list, {event | negative << 31, weight bits}; launch_hist_list then
// histograms the lists, reading each event's codes from an event-major copy
// of the code matrix (launch_transpose_codes).  Lists need n < 2^31 and at
// most kListMaxSlots slots.
constexpr int kListMaxSlots = 64;
constexpr int64_t kListMaxEvents = ((int64_t)1 << 31) - 1;
// features per workgroup of the list pass it is built for (multiples of 4:
// a workgroup reads an entry's codes as words)
constexpr int kListFpgSizes[] = {4, 8, 12, 20, 28, 36, 40};
bool list_fpg_supported(int f);
// bytes per event of the event-major copy (d rounded up to 16, 32 or 64,
// then to a multiple of 64, so that a row is whole 16-byte words and never
// straddles a 64-byte memory segment), and the copy's size (events rounded
// up to 256)
int list_row_bytes(int d);
size_t list_codes_bytes(int64_t n, int d);
hipError_t launch_transpose_codes(const uint8_t *xb, int64_t ldb, int64_t n, int d, uint8_t *xr,
                                  hipStream_t s);

struct ListShape {
    int fpg;            // features per workgroup
    int groups;         // ceil(d / fpg)
    int parts;          // workgroups per feature group that share the lists' entries (> lists)
    int lists;          // histogrammed lists of the layer
    int per_xcd;        // workgroups per XCD
    int blocks;         // kXcds * per_xcd
    int copies;         // LDS copies of the rows (lane l adds into copy l % copies)
    int copy_stride;    // bytes between copies
    size_t lds_bytes;   // dynamic LDS per workgroup
};
// fpg / parts / copies: overrides (0 = the planner's choice).
ListShape plan_list_histogram(int d, int lists, int cu_count, size_t max_lds, int fpg,
                              int parts, int copies);

// Routing of layer `layer` in [1, 6] with list output.  node_in: ids of
// layer - 1 (null at layer 1: all events at the root); node_out receives the
// ids of the layer for round_up(n, 8) events.  w, vsign as for
// launch_histogram.  lmode kCutSibling: one child per parent is listed, the
// lighter one in the parents' summed prefix rows hparent [2^(layer-1)][d]
// [B][2] (lside[k] = 1: the right child of parent k), list k = parent k;
// kCutStopped (missing values): that child in list 2k and the events that
// stop at parent k in list 2k + 1; kCutPlain: every node of the layer.
// cap_prev: bounds on the on-grid sampled events per node of layer - 1
// (launch_hist_list's cnt_out of that layer; null at layer 1: cap_root for
// the root); cursor [lists] (zeroed): receives the entries per list; lstart
// / lcap [lists]: each list's range in `list` (at most cap_root entries with
// hparent, else 2 cap_root); small: the layer's side histogram
// [2^layer][d][B][2].
hipError_t launch_route_list(const uint8_t *xb, int64_t ldb, int64_t n, int d, int n_bins,
                             const uint8_t *node_in, uint8_t *node_out, const float *w,
                             const uint8_t *vsign, const ParentCuts &pc, int layer, bool miss,
                             int lmode, const uint64_t *hparent, int scale,
                             const uint32_t *cap_prev,
                             uint32_t cap_root, uint32_t *cursor,
                             uint32_t *lstart, uint32_t *lcap, uint32_t *lside, uint2 *list,
                             double *small, uint32_t *sany, int *err, hipStream_t s);
// (sany: set non-zero when a weight goes to small)
// Histograms of the ls.lists lists of launch_route_list (lmode as there,
// lside from the route pass) into prefix-summed partials [ls.parts][d][B]
// [2], with lchunks [ls.lists] = {first part, parts | right child
// histogrammed << 31} for the cut scan.  cnt_out (optional) [2^layer]
// receives bounds on the on-grid sampled events of every node of the layer
// (the next layer's cap_prev): a listed node's entries, the other child of
// a parent its capacity minus the listed child's entries (and minus the
// events that stopped at the parent).
hipError_t launch_hist_list(const ListShape &ls, int lmode, const uint2 *list,
                            const uint32_t *lstart, const uint32_t *lcap, const uint32_t *cursor,
                            const uint32_t *lside, const uint8_t *xr, int d, int n_bins,
                            bool signed_w, int scale, uint2 *lchunks, uint64_t *partial, int *err,
                            uint32_t *cnt_out, hipStream_t s);

// Forest traversal.  cuts: [T][2^D-1] packed (feature | bin << 8), for the
// general kernel; nodes: [T][16] for depth <= kApplyShallowDepth, for heap
// node k + 1 word k = feature * apply_node_stride (the LDS row offset in the
// launch's code tile) and word 8 + k = (256 - bin) * 0x10001.
constexpr int kApplyShallowDepth = 3;
struct ApplyShape {
    bool shallow;          // depth <= kApplyShallowDepth: apply_shallow_kernel
    bool missing;          // missing values: boost weights of every node per tree (heap
                           // order) and the missing code stops an event at its node
    int threads;
    int blocks;
    int trees_per_chunk;   // trees whose leaf values (and cuts) are staged in LDS at once
    int d_used;
    size_t lds_bytes;
};
ApplyShape plan_apply(int64_t n, int d_used, int n_trees, int depth, bool missing,
                      int cu_count, size_t max_lds, int threads);
inline int apply_node_stride(const ApplyShape &as) { return 2 * as.threads + 8; }
hipError_t launch_apply(const ApplyShape &as, const uint8_t *xb, int64_t ldb, int64_t n,
                        const uint16_t *cuts, const uint32_t *nodes, const double *leaves,
                        int n_trees, int depth, double f0, float *prob, double *score,
                        hipStream_t s);

// Per-event importance [d_out][ldi] (float64) of binned events: the gains of
// the nodes on each event's path summed per cut feature, tree by tree.
// cuts: [T][2^D-1] packed (feature | bin << 8); gains: [T][2^D-1].
ApplyShape plan_importance(int64_t n, int d_used, int n_trees, int depth, bool missing,
                           int cu_count, size_t max_lds);
hipError_t launch_importance(const ApplyShape &as, const uint8_t *xb, int64_t ldb, int64_t n,
                             const uint16_t *cuts, const double *gains, int n_trees, int depth,
                             double *imp, int64_t ldi, int d_out, hipStream_t s);

// Traversal of float32 events [d][ldx] with value thresholds.  Forests of
// depth <= kApplyShallowDepth without missing values (as.shallow) take the
// binned shallow traversal with its code tile staged from the values:
// ftab = [d_used + 1] offsets, then per feature the ascending distinct
// thresholds its cuts test (float bits), ftab_words words in all (table_bytes
// of LDS); fnodes = node records as for the binned traversal (stride
// apply_node_stride(as)) with word 8 + k = (256 - c') * 0x10001, c' the rank
// (from 1) of the node's threshold among its feature's.  Other forests walk
// rec: [T][2^D-1] (feature, float bits of the threshold) per heap node.
ApplyShape plan_apply_float(int64_t n, int d_used, int n_trees, int depth, bool missing,
                            int cu_count, size_t max_lds, int threads, size_t table_bytes);
hipError_t launch_apply_float(const ApplyShape &as, const float *x, int64_t ldx, int64_t n,
                              const uint2 *rec, const uint32_t *fnodes, const uint32_t *ftab,
                              int ftab_words, const double *leaves, int n_trees, int depth,
                              double f0, float *prob, double *score, hipStream_t s);

// Equal-frequency boundaries on the device: for every feature the value of
// rank floor(k n / B), k = 1 .. B - 1, from a radix sort of the feature's
// values (batches of features whose keys together stay <= kQuantileBatchKeys).
constexpr int64_t kQuantileBatchKeys = (int64_t)1 << 27;
struct QuantileScratch {
    int batch_features;   // features sorted together
    size_t key_elems;     // 64-bit keys per buffer (two buffers)
    size_t temp_bytes;    // sort scratch
};
int quantile_batch_features(int64_t n, int d);
hipError_t quantile_scratch(int64_t n, int d, QuantileScratch *qs);
// x: device float32 [d][ldx]; bounds: device float32 [d][n_bins - 1], over
// the non-NaN values of each feature; nan_count: device [d] scratch; err
// receives kErrNan if a value is NaN and n_bins > kMissingCode.
hipError_t launch_quantile_boundaries(const float *x, int64_t ldx, int64_t n, int d, int n_bins,
                                      const QuantileScratch &qs, uint64_t *keys_a,
                                      uint64_t *keys_b, void *temp,
                                      unsigned long long *nan_count, float *bounds, int *err,
                                      hipStream_t s);

hipError_t launch_encode(const float *x, int64_t ldx, int64_t n, int d, const float *bounds,
                         int n_bins, uint8_t *xb, int64_t ldb, int *err, hipStream_t s);

}  // namespace fbdt
