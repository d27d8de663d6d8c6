// HIP kernels of libfbdt for gfx950 (CDNA4, wave64).
//
// The fit and apply path of FastBDT (Keck, arXiv:1609.06119):
//   tree_prep      score update + gradient re-weighting + sub-sample (sections 1.3, 1.4)
//   hist           one pass over the sample builds the signal/background
//                  histograms of all nodes and features of a layer (sections 1.1, 2.1),
//                  routing every event from the previous layer on the way (Fig. 1)
//   best_cuts      cumulative histograms, separation gain, best cut (section 1.1)
//   leaf           last routing + Newton-step terminal boost weights (section 1.3)
//   apply          forest traversal and sigmoid of the summed boost weights (section 1.3)
//   encode         equal-frequency bin codes from boundaries (section 2.2)
//
// Data layout in HBM: binned features are feature-major uint8 rows (row
// stride ldb, a multiple of 16), so a wavefront reads 64 consecutive events
// of one feature as one 256-byte run; per-event state (node id uint8, signed
// float32 weight, float64 score) lives in separate arrays.
#include "fbdt_internal.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdlib>
#include <cstdint>

namespace fbdt {
namespace {

constexpr int kWave = 64;
constexpr int kHistE = 8;      // events per thread and step of the histogram pass

// Workgroup barrier that orders LDS only: this wavefront's LDS operations
// complete before it (s_waitcnt lgkmcnt(0)), while its global loads and
// stores may stay in flight across it (the compiler still waits for a
// loaded register where it is used).  For barriers that publish LDS data
// only, so that prefetched event data keeps arriving and stores keep draining.
__device__ __forceinline__ void lds_barrier() {
    __asm__ volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// SplitMix64 (Steele, Lea & Flood, OOPSLA 2014): output number k (0-based)
// of the generator seeded with `seed` mixes the state seed + (k + 1) * gamma.
__device__ __forceinline__ uint64_t splitmix64_at(uint64_t seed, uint64_t k) {
    uint64_t z = seed + (k + 1ull) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// Event i of tree t is in the sub-sample iff the top 53 bits of output
// t * n + i, over 2^53, are below alpha (section 1.4).
__device__ __forceinline__ bool in_subsample(uint64_t seed, int tree, int64_t n, int64_t i,
                                             double alpha) {
    const uint64_t k = (uint64_t)tree * (uint64_t)n + (uint64_t)i;
    const double u = (double)(splitmix64_at(seed, k) >> 11) * 0x1.0p-53;
    return u < alpha;
}

// Pseudo-response of the binomial deviance with F half the log-odds
// (section 1.3, Friedman's two-class LK_TreeBoost): 2y / (1 + exp(2yF)).
__device__ __forceinline__ double pseudo_response(double yf, double F) {
    return 2.0 * yf / (1.0 + exp(2.0 * yf * F));
}

// Weighted Gini impurity G(s, b) = s b / (s + b), zero for an empty side.
__device__ __forceinline__ double gini(double s, double b) {
    const double t = s + b;
    return t == 0.0 ? 0.0 : (s * b) / t;
}

template <typename T>
__device__ __forceinline__ T load_agent(const T *p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------------
__global__ void fill_u32_kernel(uint32_t *p, uint32_t value, size_t count) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < count;
         i += (size_t)gridDim.x * blockDim.x)
        p[i] = value;
}

// ---------------------------------------------------------------------------
// Label/weight checks and per-class weight sums (deterministic order:
// fixed grid, grid-stride per thread, fixed reduction tree).
__global__ __launch_bounds__(256) void validate_kernel(const int8_t *__restrict__ y,
                                                       const float *__restrict__ v, int64_t n,
                                                       double *__restrict__ class_partial,
                                                       int *__restrict__ err) {
    // per block: signal total, background total, sum of |v|
    double s = 0.0, b = 0.0, a = 0.0;
    int e = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int yi = y[i];
        const float vi = v ? v[i] : 1.0f;
        if (yi != 1 && yi != -1) e |= kErrLabel;
        if (!isfinite(vi)) e |= kErrWeight;
        if (vi < 0.0f) e |= kNegWeights;
        if (yi > 0)
            s += (double)vi;
        else if (yi < 0)
            b += (double)vi;
        a += fabs((double)vi);
    }
    for (int off = kWave / 2; off > 0; off >>= 1) {
        s += __shfl_down(s, off);
        b += __shfl_down(b, off);
        a += __shfl_down(a, off);
    }
    __shared__ double ws[256 / kWave][3];
    const int lane = threadIdx.x % kWave, wid = threadIdx.x / kWave;
    if (lane == 0) {
        ws[wid][0] = s;
        ws[wid][1] = b;
        ws[wid][2] = a;
    }
    if (e) atomicOr(err, e);
    __syncthreads();
    if (threadIdx.x == 0) {
        double ts = 0.0, tb = 0.0, ta = 0.0;
        for (int k = 0; k < (int)(blockDim.x / kWave); ++k) {
            ts += ws[k][0];
            tb += ws[k][1];
            ta += ws[k][2];
        }
        class_partial[3 * blockIdx.x] = ts;
        class_partial[3 * blockIdx.x + 1] = tb;
        class_partial[3 * blockIdx.x + 2] = ta;
    }
}

// F0 = 1/2 ln(sum of signal weight / sum of background weight).
__global__ __launch_bounds__(256) void initial_score_kernel(const double *__restrict__ cp,
                                                            int nblocks, double *__restrict__ f0,
                                                            int *__restrict__ err) {
    __shared__ double sh[256][3];
    double s = 0.0, b = 0.0, a = 0.0;
    for (int k = threadIdx.x; k < nblocks; k += blockDim.x) {
        s += cp[3 * k];
        b += cp[3 * k + 1];
        a += cp[3 * k + 2];
    }
    sh[threadIdx.x][0] = s;
    sh[threadIdx.x][1] = b;
    sh[threadIdx.x][2] = a;
    __syncthreads();
    for (int off = blockDim.x / 2; off > 0; off >>= 1) {
        if ((int)threadIdx.x < off) {
            sh[threadIdx.x][0] += sh[threadIdx.x + off][0];
            sh[threadIdx.x][1] += sh[threadIdx.x + off][1];
            sh[threadIdx.x][2] += sh[threadIdx.x + off][2];
        }
        __syncthreads();
    }
    if (threadIdx.x == 0) {
        const double ts = sh[0][0], tb = sh[0][1];
        if (!(ts > 0.0 && tb > 0.0))
            atomicOr(err, kErrClass);
        else
            f0[0] = 0.5 * log(ts / tb);
        f0[1] = sh[0][2];   // sum of |v|: bounds every histogram sum
    }
}

// ---------------------------------------------------------------------------
// Sum of the workgroup partials of the leaf pass in a fixed order by a
// workgroup of kLeafReduceThreads threads, and the boost weights
// eta * num / den (0 when den = 0) into s_leaf[0, nleaf).  Every thread of
// the workgroup calls it; red holds kLeafReduceThreads doubles of LDS.  The
// same order everywhere gives the same weights in every workgroup that calls
// it.  With nv = 2 nleaf <= 64 values: lane l of wavefront w takes value
// l % nv and stripe s = w (64 / nv) + l / nv of the S = 16 (64 / nv) stripes,
// sums blocks s, s + S, ... in order, the wavefront adds its stripes with
// xor shuffles (fixed tree), and 16 wavefront sums are added in order.
// Larger nv: thread t takes value t % nv over stripes of kLeafReduceThreads
// / nv, then the stripes are added pairwise.
constexpr int kLeafReduceThreads = 1024;
// (num, den) pairs of every terminal slot of the deepest tree: with missing
// values at depth 7, 255 nodes
constexpr int kLeafSumSlots = 2 * ((2 << 7) - 1);

// With missing values (section 4.2) the slots are all nodes of the tree in
// heap order (slot k - 1 = node k) holding (num, den) of the events whose
// terminal node it is: every inner node (the first `inner` slots) adds its
// children's sums, bottom up in a fixed order, and then every slot becomes
// eta * num / den (0 where den = 0).  s[2 slot] = num, s[2 slot + 1] = den
// on entry; s[slot] = the weight on exit.
__device__ void node_sums_to_weights(double *s, int nslots, int inner, double eta) {
#pragma clang fp contract(off)
    if (threadIdx.x == 0) {
        for (int k = inner; k >= 1; --k) {   // node k's children: nodes 2k, 2k + 1
            s[2 * (k - 1)] += s[2 * (2 * k - 1)] + s[2 * (2 * k)];
            s[2 * (k - 1) + 1] += s[2 * (2 * k - 1) + 1] + s[2 * (2 * k) + 1];
        }
        for (int k = 0; k < nslots; ++k) {
            const double num = s[2 * k], den = s[2 * k + 1];
            s[k] = den == 0.0 ? 0.0 : eta * (num / den);
        }
    }
    __syncthreads();
}

__device__ void reduce_leaf_partials(const double *__restrict__ leaf_partial, int nblocks,
                                     int nleaf, double eta, double *red, double *s_leaf,
                                     int bottom_up_inner = 0) {
#pragma clang fp contract(off)
    const int nv = 2 * nleaf;
    const int t = threadIdx.x;
    if (nv <= kWave && (nv & (nv - 1)) == 0) {   // a power of two: lanes share a wavefront
        const int lane = t % kWave, wave = t / kWave;
        const int per_wave = kWave / nv;
        const int stripes = (kLeafReduceThreads / kWave) * per_wave;
        const int val = lane % nv, st = wave * per_wave + lane / nv;
        double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
        int b = st;
        for (; b + 3 * stripes < nblocks; b += 4 * stripes) {
            s0 += leaf_partial[(size_t)b * nv + val];
            s1 += leaf_partial[(size_t)(b + stripes) * nv + val];
            s2 += leaf_partial[(size_t)(b + 2 * stripes) * nv + val];
            s3 += leaf_partial[(size_t)(b + 3 * stripes) * nv + val];
        }
        for (; b < nblocks; b += stripes) s0 += leaf_partial[(size_t)b * nv + val];
        double x = (s0 + s1) + (s2 + s3);
        for (int o = nv; o < kWave; o <<= 1) x += __shfl_xor(x, o);
        if (lane < nv) red[wave * nv + lane] = x;
        lds_barrier();
        if (t < nleaf) {
            double num = 0.0, den = 0.0;
            for (int w = 0; w < kLeafReduceThreads / kWave; ++w) {
                num += red[w * nv + 2 * t];
                den += red[w * nv + 2 * t + 1];
            }
            if (bottom_up_inner) {
                s_leaf[2 * t] = num;
                s_leaf[2 * t + 1] = den;
            } else {
                s_leaf[t] = den == 0.0 ? 0.0 : eta * (num / den);
            }
        }
        lds_barrier();
        if (bottom_up_inner) node_sums_to_weights(s_leaf, nleaf, bottom_up_inner, eta);
        return;
    }
    int stripes = 1;   // a power of two
    while (2 * stripes * nv <= kLeafReduceThreads) stripes *= 2;
    if (t < stripes * nv) {
        const int val = t % nv, st = t / nv;
        double s0 = 0.0, s1 = 0.0, s2 = 0.0, s3 = 0.0;
        int b = st;
        for (; b + 3 * stripes < nblocks; b += 4 * stripes) {
            s0 += leaf_partial[(size_t)b * nv + val];
            s1 += leaf_partial[(size_t)(b + stripes) * nv + val];
            s2 += leaf_partial[(size_t)(b + 2 * stripes) * nv + val];
            s3 += leaf_partial[(size_t)(b + 3 * stripes) * nv + val];
        }
        for (; b < nblocks; b += stripes) s0 += leaf_partial[(size_t)b * nv + val];
        red[t] = (s0 + s1) + (s2 + s3);
    }
    __syncthreads();
    // stripes (a power of two) added pairwise: red[st] += red[st + half]
    for (int half = stripes / 2; half >= 1; half >>= 1) {
        if (t < half * nv) red[t] += red[t + half * nv];
        __syncthreads();
    }
    if (t < nleaf) {
        const double num = red[2 * t], den = red[2 * t + 1];
        if (bottom_up_inner) {
            s_leaf[2 * t] = num;
            s_leaf[2 * t + 1] = den;
        } else {
            s_leaf[t] = den == 0.0 ? 0.0 : eta * (num / den);
        }
    }
    __syncthreads();
    if (bottom_up_inner) node_sums_to_weights(s_leaf, nleaf, bottom_up_inner, eta);
}

// ---------------------------------------------------------------------------
// One elementwise pass per tree: add the previous tree's boost weight to F
// (or set F = F0 for the first tree), then the histogram weight of every
// event: fl32(v |y~|) if sampled else 0, class in the sign bit, and (yts)
// the pseudo-response y~ of the sampled events, 0 for the others.  The
// previous tree's boost weights come either from the model (leaf_prev) or
// straight from the leaf pass partials (leaf_partial, depth <= 4), which
// every workgroup sums itself in the fixed order of leaf_finalize_kernel;
// workgroup 0 then records them in the model (leaf_rec).
struct PrepStep {
    int yv;
    uint32_t leaf;
    float v;
    double F;
    bool sampled;   // depends on (seed, tree, i) only: decided while the loads fly
};

__global__ __launch_bounds__(kLeafReduceThreads) void tree_prep_kernel(
    const int8_t *__restrict__ y, const float *__restrict__ v, double *__restrict__ F,
    const double *__restrict__ f0, const uint8_t *__restrict__ leaf_node,
    const double *__restrict__ leaf_prev, const double *__restrict__ leaf_partial,
    int lblocks, double eta, double *__restrict__ leaf_rec, int depth, bool missing, int64_t n,
    uint64_t seed, int tree, double alpha, float *__restrict__ w, double *__restrict__ yts,
    double *__restrict__ score_out, int64_t xcd_events) {
    __shared__ double red[kLeafReduceThreads];
    __shared__ double s_leaf[kLeafSumSlots];
    // boost weights of the terminal nodes: the leaves (heap ids from 2^D), or
    // with missing values every node (heap ids from 1)
    const unsigned nleaf = 1u << depth;
    const unsigned nslots = missing ? 2u * nleaf - 1u : nleaf;
    const unsigned first_id = missing ? 1u : nleaf;
    const bool have_leaf = leaf_prev || leaf_partial;
    const bool read_F = have_leaf || !f0;
    // the workgroups on XCD x = blockIdx % 8 take the events [x R, (x + 1) R)
    const int64_t xlo = (int64_t)(blockIdx.x % kXcds) * xcd_events;
    const int64_t xend = min(n, xlo + xcd_events);
    const int64_t stride = (int64_t)(gridDim.x / kXcds) * blockDim.x;
    int64_t ia = xlo + (int64_t)(blockIdx.x / kXcds) * blockDim.x + threadIdx.x;
    // one event per thread and step; the first step's loads are in flight
    // while the boost weights are summed, later steps are loaded one ahead
    const bool need_sample = w || yts;
    auto load = [&](PrepStep &st, int64_t i) {
        st.yv = y[i];
        st.v = v ? v[i] : 1.0f;
        st.leaf = have_leaf ? (uint32_t)leaf_node[i] : 0u;
        st.F = read_F ? F[i] : 0.0;
        st.sampled = need_sample && in_subsample(seed, tree, n, i, alpha);
    };
    PrepStep A, B;
    if (ia < xend) load(A, ia);
    if (leaf_partial) {
        reduce_leaf_partials(leaf_partial, lblocks, (int)nslots, eta, red, s_leaf,
                             missing ? (int)nleaf - 1 : 0);
        if (blockIdx.x == 0 && leaf_rec && threadIdx.x < nslots)
            leaf_rec[threadIdx.x] = s_leaf[threadIdx.x];
    } else if (leaf_prev) {
        for (unsigned t = threadIdx.x; t < nslots; t += blockDim.x) s_leaf[t] = leaf_prev[t];
        lds_barrier();
    }
    const double f0v = (f0 && !have_leaf) ? *f0 : 0.0;
    auto step = [&](const PrepStep &st, int64_t i) {
        double Fi;
        if (have_leaf) {
            unsigned li = st.leaf - first_id;
            if (li >= nslots) li = 0;  // unreachable: terminal ids come from the leaf pass
            Fi = st.F + s_leaf[li];
            F[i] = Fi;
        } else if (f0) {
            Fi = f0v;
            F[i] = Fi;
        } else {
            Fi = st.F;
        }
        if (score_out) score_out[i] = Fi;
        if (w || yts) {
            const double yf = (double)st.yv;
            const double yt = pseudo_response(yf, Fi);
            const bool sampled = st.sampled;
            if (w) {
                const double vi = (double)st.v;
                // |fl32(v |y~|)| with the class in the sign bit (a negative
                // v's sign travels in the separate sign bytes of the fit)
                const float wi = sampled ? fabsf((float)(vi * fabs(yt))) : 0.0f;
                w[i] = yf > 0.0 ? wi : -wi;
            }
            if (yts) yts[i] = sampled ? yt : 0.0;
        }
    };
    if (ia < xend) {
        for (;;) {
            const int64_t ib = ia + stride;
            if (ib < xend) load(B, ib);
            step(A, ia);
            if (ib >= xend) break;
            ia = ib + stride;
            if (ia < xend) load(A, ia);
            step(B, ib);
            if (ia >= xend) break;
        }
    }
}

// ---------------------------------------------------------------------------
// Candidate cuts of a layer: entry e = j * S + q of node k holds the best cut
// (gain, bin) of feature j among the bins of slice q (S slices per feature,
// bins rising with q), so that the entry order is the (feature, bin) order.
// The best candidate of a node (gain highest, then lowest entry: lowest
// feature, then lowest bin) is found by one wavefront; lane 0 returns it.  An
// unusable result (no finite gain) falls back to feature 0 and reports it.
// (The fit's routed passes take their cuts from the best-cut keys below.)
struct CandSet {
    const double *gain;   // [nodes][E]
    const int *cut;       // [nodes][E]
    int d;                // features
    int S;                // slices per feature; E = d * S entries per node
};

constexpr int kCutSlice = 31;   // cuts per slice (the cut scan's workgroups)

__device__ __forceinline__ void node_best(const CandSet &cs, int k, int lane, int *bf, int *bc,
                                          double *bg, bool *ok) {
    const int E = cs.d * cs.S;
    double g = -INFINITY;
    int idx = 0x7fffffff, c = 1;
    // each lane visits its entries in rising order: a strict > keeps the lowest
    for (int e = lane; e < E; e += kWave) {
        const double x = cs.gain[(size_t)k * E + e];
        if (x > g) {
            g = x;
            idx = e;
            c = cs.cut[(size_t)k * E + e];
        }
    }
#pragma unroll
    for (int off = kWave / 2; off > 0; off >>= 1) {
        const double og = __shfl_xor(g, off);
        const int oi = __shfl_xor(idx, off);
        const int oc = __shfl_xor(c, off);
        if (og > g || (og == g && oi < idx)) {
            g = og;
            idx = oi;
            c = oc;
        }
    }
    const int j = idx < E ? idx / cs.S : cs.d;
    *ok = j < cs.d && c >= 1 && c <= 255;
    *bf = *ok ? j : 0;
    *bc = *ok ? c : 1;
    *bg = g;
}

// Best cut of a node as one 64-bit key, so that the cut scan can take the
// maximum over all of a node's candidates with atomicMax: the gain's bits
// mapped to an unsigned order (sign bit set for non-negative values, every
// bit flipped for negative ones; -0 taken as +0), with the low 16 bits
// replaced by 0xffff - (256 j + c), so that the higher gain wins, then the
// lower (feature, bin).  Gains that differ only in those 16 mantissa bits
// (2^-36 relative) count as tied.  A finite or +inf gain gives a non-zero
// key; 0 means that the node has no candidate.
__device__ __forceinline__ unsigned long long cut_key(double g, int j, int c) {
    const unsigned long long u = (unsigned long long)__double_as_longlong(g == 0.0 ? 0.0 : g);
    const unsigned long long o = (u >> 63) ? ~u : (u | (1ull << 63));
    return (o & ~0xffffull) | (0xffffull - (unsigned long long)(j * 256 + c));
}

// Feature and bin of a key; an absent or unusable key falls back to feature
// 0, bin 1 and reports it (ok = false).
__device__ __forceinline__ void key_cut(unsigned long long key, int d, int *bf, int *bc, bool *ok) {
    const int jc = 0xffff - (int)(key & 0xffffull);
    const int j = jc >> 8, c = jc & 0xff;
    *ok = key != 0ull && j < d && c >= 1;
    *bf = *ok ? j : 0;
    *bc = *ok ? c : 1;
}

// The key slots of parent k (one per XCD), loaded so that a kernel can
// issue them early, and their maximum, the parent's key.
struct KeySlots {
    unsigned long long v[kXcds];
};

__device__ __forceinline__ void key_load(const unsigned long long *keys, int k, KeySlots &r) {
#pragma unroll
    for (int x = 0; x < kXcds; ++x) r.v[x] = keys[((size_t)k * kXcds + x) * kKeyStride];
}

__device__ __forceinline__ unsigned long long key_max(const KeySlots &r) {
    unsigned long long m = r.v[0];
#pragma unroll
    for (int x = 1; x < kXcds; ++x) m = max(m, r.v[x]);
    return m;
}

// Cut of parent k of a routed pass from its key slots into the cut table.
__device__ __forceinline__ void parent_cut(const KeySlots &r, int k, int d, uint8_t *s_cf,
                                           uint8_t *s_cc, int &eflag) {
    int bf, bc;
    bool ok;
    key_cut(key_max(r), d, &bf, &bc, &ok);
    s_cf[k] = (uint8_t)bf;
    s_cc[k] = (uint8_t)bc;
    if (!ok) eflag |= kErrRoute;
}

// Parent k's cut recorded in the model once the cut table is in LDS:
// feature and bin; returns the gain to record, that of the candidate of the
// slice that holds the cut (a load that the caller stores at its end, so
// that no wavefront waits for it).
__device__ __forceinline__ double record_parent_cut(const uint8_t *s_cf, const uint8_t *s_cc,
                                                    int k, int d, int S, const double *cand_gain,
                                                    uint8_t *rec_f, uint8_t *rec_c) {
    const int f = s_cf[k], c = s_cc[k];
    rec_f[k] = (uint8_t)f;
    rec_c[k] = (uint8_t)c;
    return cand_gain[((size_t)k * d + f) * S + (c - 1) / kCutSlice];
}

// Cuts of n_nodes nodes from their candidates (one wavefront per node).
__global__ __launch_bounds__(64) void select_cuts_kernel(const double *__restrict__ cand_gain,
                                                         const int *__restrict__ cand_cut, int d,
                                                         int S, uint8_t *__restrict__ out_f,
                                                         uint8_t *__restrict__ out_c,
                                                         double *__restrict__ out_g) {
    int bf, bc;
    double bg;
    bool ok;
    node_best(CandSet{cand_gain, cand_cut, d, S}, blockIdx.x, threadIdx.x, &bf, &bc, &bg, &ok);
    if (threadIdx.x == 0) {
        out_f[blockIdx.x] = (uint8_t)bf;
        out_c[blockIdx.x] = (uint8_t)bc;
        out_g[blockIdx.x] = bg;
    }
}

// ---------------------------------------------------------------------------
// Layer histogram.  Workgroup (chunk p, feature group g, node group h) keeps
// H[node in h][feature in g][bin][class] in LDS as 64-bit fixed point
// (weight * 2^scale), adds every counted event of its event chunk with a
// 64-bit integer LDS atomic, and writes its partial histogram once at the
// end; integer sums are exact, so the result is independent of the order of
// the adds, and best_cuts sums the chunk partials.
//
// Each thread handles kHistE consecutive events per step and loads the next
// step's weights, node ids, routing rows and the codes of the group's FPG
// features before it adds the current step's events.  Per event it forms
// once its node of this layer (routing), the LDS offset of its (node, class)
// counters, the fixed-point value and whether it counts; one branch per
// event then covers its FPG atomics, whose feature-row offsets are
// immediates of the LDS instruction.
//
// Routed mode computes every event's node of this layer from its parent
// (layer - 1) and the parent's cut on the way; the first feature group
// stores the new ids.  With NP > 0 (NP = number of parents) the code rows of
// the parents' cut features are loaded for the step up front, so routing
// costs no dependent load; with NP = 0 each event's routing code is
// gathered after its parent id arrives.  The fit routes layers with more
// than kRoutedMaxParents parents by a pass of its own (route_layer_kernel)
// and histograms them with ROUTED = false from the new ids.  MISS (routed
// passes of fits with missing values) adds the stops at the missing code
// and histograms both children; otherwise layers below the root histogram
// the left children only (sibling subtraction), in both modes.
//
// An LDS row of (node, feature) holds 256 bins x 2 classes (4 KiB) whatever
// n_bins; codes >= n_bins land in bins that are checked at the end and
// reported as an error.  The last feature group may run past feature d - 1:
// its missing features load the codes of feature d - 1 and add them into
// rows that are never written out, so the inner loop has no feature test.
// Inclusive prefix sum of a 64-bit value over the 64 lanes of a wavefront
// with DPP lane moves (no LDS round trip): a Hillis-Steele scan within each
// row of 16 lanes (row_shr 1, 2, 4, 8), then the last lane of row 0 and 2
// added to rows 1 and 3 (row_bcast 15) and the last lane of row 1 to rows 2
// and 3 (row_bcast 31).  Lanes that a move does not reach receive 0.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ unsigned long long dpp_u64(unsigned long long x) {
    const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)x, CTRL, ROW_MASK, 0xf, true);
    const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(x >> 32), CTRL, ROW_MASK, 0xf,
                                               true);
    return ((unsigned long long)(uint32_t)hi << 32) | (uint32_t)lo;
}

__device__ __forceinline__ unsigned long long wave_inclusive_scan_u64(unsigned long long x) {
    x += dpp_u64<0x111, 0xf>(x);   // row_shr:1
    x += dpp_u64<0x112, 0xf>(x);   // row_shr:2
    x += dpp_u64<0x114, 0xf>(x);   // row_shr:4
    x += dpp_u64<0x118, 0xf>(x);   // row_shr:8
    x += dpp_u64<0x142, 0xa>(x);   // row_bcast:15 into rows 1, 3
    x += dpp_u64<0x143, 0xc>(x);   // row_bcast:31 into rows 2, 3
    return x;
}

constexpr int kRow = 256 * 2;                        // counters per LDS row
constexpr int kRowBytes = kRow * (int)sizeof(uint64_t);

__device__ __forceinline__ uint32_t byte8(const uint2 &v, int e) {
    const uint32_t w = e < 4 ? v.x : v.y;
    return (w >> (8 * (e & 3))) & 0xffu;
}

template <int NP, int FPG>
struct HistStep {
    uint32_t w[kHistE];               // weight bits (class in the sign bit)
    uint2 node;                       // parent ids (routed, layer >= 2) or node ids
    uint2 vs;                         // 1 where the event's weight is negative (signed fits)
    uint2 rows[NP > 0 ? NP : 1];      // codes of the parents' cut features
    uint2 codes[FPG];                 // codes of the group's features
};

// Uniform per-workgroup arguments of the histogram pass.
struct HistArgs {
    const uint8_t *xb;
    int64_t ldb, n;
    int d, nbins, layer, nodes, half, j0, nf, k0, nk, scale;
    int jstep;                        // the group's features: j0, j0 + jstep, ... (nf of them)
    bool miss;                        // n_bins <= kMissingCode: code kMissingCode is missing
    bool sib;                         // left children only (right = parent - left)
    uint32_t tau_bits;                // bits of the smallest weight on the fixed-point grid
    const uint8_t *node_in;
    uint8_t *node_out;
    const float *w;
    const uint8_t *vsign;             // [padded n] 1 = negative event weight (signed fits)
    double *small;
};

// codes of the parents' cut features (the cut table must be in LDS)
template <bool ROUTED, int NP, int FPG, bool SIGNED, bool MISS>
__device__ __forceinline__ void hist_load_rows(HistStep<NP, FPG> &st, const HistArgs &a,
                                               const uint8_t *s_cf, int64_t i0) {
    if (ROUTED && NP > 0 && a.layer >= 1) {
        // rows are padded to ldb >= i0 + kHistE: always in bounds
#pragma unroll
        for (int kk = 0; kk < (NP > 0 ? NP : 1); ++kk)
            st.rows[kk] = *reinterpret_cast<const uint2 *>(
                a.xb + (int64_t)min((int)s_cf[kk], a.d - 1) * a.ldb + i0);
    }
}

// The per-event arrays (weights, node ids) are padded to a multiple of
// kHistE with zero weights, and code rows to ldb >= that padding, so every
// step loads kHistE whole events; padded events weigh 0 and count nowhere.
template <bool ROUTED, int NP, int FPG, bool SIGNED, bool MISS>
__device__ __forceinline__ void hist_load(HistStep<NP, FPG> &st, const HistArgs &a,
                                          const uint8_t *s_cf, int64_t i0, bool with_rows) {
    const uint4 x = reinterpret_cast<const uint4 *>(a.w + i0)[0];
    const uint4 y = reinterpret_cast<const uint4 *>(a.w + i0)[1];
    st.w[0] = x.x; st.w[1] = x.y; st.w[2] = x.z; st.w[3] = x.w;
    st.w[4] = y.x; st.w[5] = y.y; st.w[6] = y.z; st.w[7] = y.w;
    if (!ROUTED || a.layer >= 2) st.node = *reinterpret_cast<const uint2 *>(a.node_in + i0);
#pragma unroll
    for (int ff = 0; ff < FPG; ++ff)
        st.codes[ff] = *reinterpret_cast<const uint2 *>(
            a.xb + (int64_t)min(a.j0 + ff * a.jstep, a.d - 1) * a.ldb + i0);
    if (SIGNED) st.vs = *reinterpret_cast<const uint2 *>(a.vsign + i0);
    if (with_rows) hist_load_rows<ROUTED, NP, FPG, SIGNED, MISS>(st, a, s_cf, i0);
}

template <bool ROUTED, int NP, int FPG, bool SIGNED, bool MISS>
__device__ __forceinline__ void hist_add(const HistStep<NP, FPG> &st, const HistArgs &a,
                                         uint64_t *lds, bool writer, const uint8_t *s_cf,
                                         const uint8_t *s_cc, const uint32_t (&cut)[4],
                                         int64_t i0, int &eflag) {
    // Per event: slot = index of the histogrammed node within the group
    // (>= nk: not this group's), nl = node of this layer - nodes (side
    // histogram index), counted = the event's node is histogrammed here.
    // Routed passes below the root with sib histogram the left child of
    // every parent only (slot = parent index); the right child's fixed-point
    // histogram is parent - left.  Without sib (fits with missing values,
    // where events that stop at a parent are in its histograms but in
    // neither child's) both children are histogrammed.  Weights below the
    // grid go to the side histogram of every node, left or right.
    uint32_t slot[kHistE], nl[kHistE];
    bool counted[kHistE];
    uint32_t bad = 0u;
    if (!ROUTED) {
        // ids of this layer; with sib the left child 2k is histogrammed in
        // slot k and the right child is parent - left; ids below the layer
        // (stopped earlier) fall outside every slot
#pragma unroll
        for (int e = 0; e < kHistE; ++e) {
            const uint32_t node = byte8(st.node, e);
            nl[e] = node - (uint32_t)a.nodes;
            slot[e] = (a.sib ? nl[e] >> 1 : nl[e]) - (uint32_t)a.k0;
            counted[e] = !a.sib | ((nl[e] & 1u) == 0u);
        }
    } else if (a.layer == 0) {
#pragma unroll
        for (int e = 0; e < kHistE; ++e) {
            nl[e] = 0u;
            slot[e] = 0u;
            counted[e] = true;
        }
    } else {
        uint32_t o[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < kHistE; ++e) {
            uint32_t par, k, code, c;
            bool stop = false;   // the event stays at its node (missing value)
            if (NP == 1) {   // layer 1: the root is the only parent
                par = 1u;
                k = 0u;
                code = byte8(st.rows[0], e);
                c = cut[0];
            } else {
                par = byte8(st.node, e);
                k = par - (uint32_t)a.half;
                if (k >= (uint32_t)a.half) {
                    // below the layer: stopped earlier at a missing value;
                    // above it: unreachable for ids written by this library
                    const bool earlier = MISS && par < (uint32_t)a.half;
                    stop = earlier;
                    bad |= earlier ? 0u : 1u;
                    k = 0u;
                    par = earlier ? par : (uint32_t)a.half;
                }
                if (NP > 0) {
                    code = byte8(st.rows[0], e);
                    c = cut[0];
#pragma unroll
                    for (int kk = 1; kk < (NP > 0 ? NP : 1); ++kk) {
                        if (k == (uint32_t)kk) {
                            code = byte8(st.rows[kk], e);
                            c = cut[kk];
                        }
                    }
                } else {
                    code = a.xb[(int64_t)min((int)s_cf[k], a.d - 1) * a.ldb + i0 + e];
                    c = s_cc[k];
                }
            }
            if (MISS) stop |= code == (uint32_t)kMissingCode;
            const uint32_t right = code >= c ? 1u : 0u;
            const uint32_t ne = stop ? par : 2u * par + right;
            o[e >> 2] |= ne << (8 * (e & 3));
            nl[e] = ne - (uint32_t)a.nodes;
            // stopped: counted nowhere; routed passes take sibling
            // subtraction exactly when no event can stop (!MISS)
            if (MISS) {
                slot[e] = stop ? 0xffffffffu : nl[e] - (uint32_t)a.k0;
                counted[e] = !stop;
            } else {
                slot[e] = k - (uint32_t)a.k0;
                counted[e] = right == 0u;
            }
        }
        // padded events get ids too, so that the next layer reads valid parents
        if (writer) *reinterpret_cast<uint2 *>(a.node_out + i0) = make_uint2(o[0], o[1]);
    }
    if (bad) eflag |= kErrRoute;
    // Counted events of this group's nodes add w * 2^scale to their
    // (node, feature, bin, class) counter: the float's 24-bit significand
    // shifted into place, exact for weights on the grid (>= tau).
    char *ldsb = reinterpret_cast<char *>(lds);
    uint32_t below = 0u;
#pragma unroll
    for (int e = 0; e < kHistE; ++e) {
        const uint32_t bits = st.w[e];
        const uint32_t ab = bits & 0x7fffffffu;
        const bool mine = slot[e] < (uint32_t)a.nk;
        if (mine && (ab - 1u) < a.tau_bits - 1u) below |= 1u << e;   // 0 < w < tau: rare
        if (mine && counted[e] && ab >= a.tau_bits) {
            const int sh = (int)(ab >> 23) - 150 + a.scale;   // >= 0 on the grid
            uint64_t fx = (uint64_t)((ab & 0x7fffffu) | 0x800000u) << sh;
            if (SIGNED && byte8(st.vs, e)) fx = 0ull - fx;   // two's complement: sums stay exact
            const uint32_t base = slot[e] * (uint32_t)(FPG * kRowBytes) + ((bits >> 28) & 8u);
#pragma unroll
            for (int ff = 0; ff < FPG; ++ff) {
                const uint32_t off = base + (byte8(st.codes[ff], e) << 4);
                atomicAdd(reinterpret_cast<uint64_t *>(ldsb + off) + ff * kRow, fx);
            }
        }
    }
    if (below) {   // weights below the grid: float64 side histogram of the event's node
        // (indices stay compile-time constants so that the step stays in registers)
#pragma unroll
        for (int e = 0; e < kHistE; ++e) {
            if ((below >> e) & 1u) {
                const uint32_t bits = st.w[e];
                double wa = (double)__uint_as_float(bits & 0x7fffffffu);
                if (SIGNED && byte8(st.vs, e)) wa = -wa;
#pragma unroll
                for (int ff = 0; ff < FPG; ++ff) {
                    const uint32_t bin = byte8(st.codes[ff], e);
                    const bool missing = a.miss & (bin == (uint32_t)kMissingCode);
                    if (ff < a.nf && bin >= (uint32_t)a.nbins && !missing) eflag |= kErrBin;
                    if (ff < a.nf && bin < (uint32_t)a.nbins) {
                        const size_t gi =
                            ((((size_t)nl[e] * a.d + a.j0 + ff * a.jstep) * a.nbins + bin) * 2) +
                            (bits >> 31);
                        atomicAdd(&a.small[gi], wa);
                    }
                }
            }
        }
    }
}

// The end of a histogram workgroup, after its adds (and an LDS barrier):
// the LDS copies are summed into copy 0, bins >= n_bins are checked to be
// empty (but for the missing code's with miss), and the rows (k, f), k < nk,
// f < nf (LDS row k * fpg + f, feature j0 + f * jstep) are written to
// out[(k0 + k) * d + j0 + f * jstep]
// [bin], the two classes of a bin in one 16-byte element: one row per
// wavefront step.  With prefix (the fit's passes) every row is written as
// inclusive prefix sums over bins, P(b) = sum of the bins <= b per class:
// summed over chunks these are the cumulative histograms, which the cut
// scan reads slice by slice.  Lane l holds bins 4l..4l+3 (both classes),
// prefix in the lane, then an exclusive scan of the lane totals across the
// wavefront.
__device__ __forceinline__ void hist_write_rows(uint64_t *lds, int copies, int copy_stride,
                                                int lds_n, int nk, int nf, int fpg, int k0,
                                                int j0, int jstep, int d, int nbins, bool miss,
                                                bool prefix, uint4 *out, int &eflag) {
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int nwaves = blockDim.x / kWave;
    if (copies > 1) {   // copy 0 += the others
        const int cs = copy_stride / 8;
        for (int t = threadIdx.x; t < lds_n; t += blockDim.x) {
            uint64_t v = lds[t];
            for (int c = 1; c < copies; ++c) v += lds[c * cs + t];
            lds[t] = v;
        }
        lds_barrier();
    }
    const int nrows = nk * nf;
    for (int rr = wave; rr < nrows; rr += nwaves) {
        const int k = rr / nf;
        const int f = rr - k * nf;
        const uint4 *src = reinterpret_cast<const uint4 *>(lds + (k * fpg + f) * kRow);
        uint4 *dst = out + ((size_t)(k0 + k) * d + j0 + f * jstep) * nbins;
        // bins >= n_bins must be empty, but for the missing code's
        for (int t = nbins + lane; t < (miss ? kMissingCode : 256); t += kWave) {
            const uint4 v = src[t];
            if (v.x | v.y | v.z | v.w) eflag |= kErrBin;
        }
        if (prefix) {   // the row is scanned in place (this wavefront's row only)
            ulonglong2 *s2 = reinterpret_cast<ulonglong2 *>(lds + (k * fpg + f) * kRow) + 4 * lane;
            ulonglong2 v[4] = {s2[0], s2[1], s2[2], s2[3]};
#pragma unroll
            for (int e = 1; e < 4; ++e) {
                v[e].x += v[e - 1].x;
                v[e].y += v[e - 1].y;
            }
            const unsigned long long xs = wave_inclusive_scan_u64(v[3].x) - v[3].x;   // exclusive
            const unsigned long long xb = wave_inclusive_scan_u64(v[3].y) - v[3].y;
#pragma unroll
            for (int e = 0; e < 4; ++e) s2[e] = make_ulonglong2(v[e].x + xs, v[e].y + xb);
        }
        for (int t = lane; t < nbins; t += kWave) dst[t] = src[t];
    }
}

template <bool ROUTED, int NP, int FPG, bool SIGNED, bool MISS>
// The arguments that the first loads need come first, so that they fit the
// kernel arguments preloaded into scalar registers at wave launch (16
// dwords): the code, weight and id arrays, the event ranges, and two packed
// words, geo = d | G << 8 | NG << 16 | chunks per XCD << 24 and mode =
// layer | sib << 3 | prefix << 4 | npg << 8 | cut slices << 16 | copies << 24.
__global__ __launch_bounds__(1024) void hist_kernel(
    const uint8_t *__restrict__ xb, const float *__restrict__ w,
    const uint8_t *__restrict__ node_in, int64_t ldb, int64_t n, int64_t chunk_events,
    int64_t xcd_events, uint32_t geo, uint32_t mode, const double *__restrict__ cand_gain,
    const unsigned long long *__restrict__ keys, int nbins, int scale, int copy_stride,
    const uint8_t *__restrict__ vsign, uint8_t *__restrict__ node_out,
    uint8_t *__restrict__ rec_f, uint8_t *__restrict__ rec_c, double *__restrict__ rec_g,
    uint64_t *__restrict__ partial, double *__restrict__ small, int *__restrict__ err,
    unsigned long long *__restrict__ tl) {
    const int d = (int)(geo & 0xffu), G = (int)((geo >> 8) & 0xffu);
    const int NG = (int)((geo >> 16) & 0xffu), cpx = (int)(geo >> 24);
    const int chunks = cpx * kXcds;
    const int layer = (int)(mode & 7u);
    const bool sib = ((mode >> 3) & 1u) != 0, prefix = ((mode >> 4) & 1u) != 0;
    const int npg = (int)((mode >> 8) & 0xffu), cslices = (int)((mode >> 16) & 0xffu);
    const int copies = (int)(mode >> 24);
    extern __shared__ uint64_t lds[];
    __shared__ uint8_t s_cf[64], s_cc[64];
    // phase timeline (measurement, tl != null): the device's constant-rate
    // clock at entry, cut table in LDS, first step added (wavefront 0), every
    // add done and partial rows written (wavefront 0), one row of
    // kTimelineStamps per workgroup
    const bool stamp = tl != nullptr && threadIdx.x == 0;
    const unsigned long long t_entry = stamp ? (unsigned long long)wall_clock64() : 0ull;
    if (tl != nullptr && threadIdx.x == blockDim.x - kWave)   // the last wavefront's entry
        tl[(size_t)blockIdx.x * kTimelineStamps + 5] = (unsigned long long)wall_clock64();

    // Consecutive work items (same event chunk, different feature groups) go
    // to the same XCD so that the chunk's node ids and weights are fetched
    // into that XCD's L2 once and re-read from there.
    const int groups = G * NG;
    const int per_xcd = cpx * groups;   // the grid is kXcds * cpx * groups workgroups
    const int q = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (q >= chunks * groups) return;
    const int p = q / groups;
    const int r = q - p * groups;
    const int h = r / G;
    const int g = r - h * G;

    HistArgs a;
    a.xb = xb;
    a.ldb = ldb;
    a.n = n;
    a.d = d;
    a.nbins = nbins;
    a.miss = nbins <= kMissingCode;
    a.layer = layer;
    a.nodes = 1 << layer;
    a.half = a.nodes >> 1;
    a.sib = layer >= 1 && sib;
    const int hnodes = a.sib ? a.half : a.nodes;   // histogrammed nodes
    // features dealt to the G groups in turn (feature j in group j % G), so
    // that features of few distinct codes, whose atomics pile onto a few
    // counters and which data sets tend to hold side by side, spread over the
    // groups instead of making one group the slowest (workload 4's eight
    // discrete features 32-39 in groups of 5: layer 0 145 -> 134 us)
    a.j0 = g;
    a.jstep = G;
    a.nf = (d - g + G - 1) / G;
    a.k0 = h * npg;
    a.nk = min(npg, hnodes - a.k0);
    a.scale = scale;
    // weights at or above tau = 2^(23 - scale) are exact multiples of 2^-scale
    a.tau_bits = __float_as_uint(ldexpf(1.0f, 23 - scale));
    a.node_in = node_in;
    a.node_out = node_out;
    a.w = w;
    a.vsign = vsign;
    a.small = small;
    const int lds_n = npg * FPG * kRow;   // counters of one copy
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    // Lane l adds into copy l % copies (copies of the same counters, each
    // shifted by a bank offset), so that lanes of one instruction whose
    // events share a bin (features with few distinct values) hit different
    // LDS addresses and banks; the copies are summed before the write-out.
    uint64_t *const lds_lane = reinterpret_cast<uint64_t *>(
        reinterpret_cast<char *>(lds) + (lane & (copies - 1)) * copy_stride);
    int eflag = 0;

    // chunk p is chunk k of XCD x's event range [x R, (x + 1) R) (the range
    // every per-event pass of the fit gives that XCD)
    const int64_t xlo = (int64_t)(p / cpx) * xcd_events;
    const int64_t start = xlo + (int64_t)(p % cpx) * chunk_events;
    const int64_t end = min(min(n, xlo + xcd_events), start + chunk_events);
    const bool writer = ROUTED && layer >= 1 && g == 0 && h == 0 && node_out != nullptr;
    const int64_t stride = (int64_t)kHistE * blockDim.x;

    // Loads in flight together: the parents' best-cut keys (the cut table of
    // a routed pass; lane k of wavefront 0 takes parent k) first, then the
    // first step's weights, node ids and codes; the step's routing rows
    // follow once the cut table is in LDS.
    const bool pwave = ROUTED && layer >= 1 && wave == 0 && lane < a.half;
    KeySlots ks;
    if (pwave) key_load(keys, lane, ks);
    HistStep<NP, FPG> A, B;
    int64_t ia = start + (int64_t)kHistE * threadIdx.x;
    if (ia < end) hist_load<ROUTED, NP, FPG, SIGNED, MISS>(A, a, s_cf, ia, false);

    {
        uint4 *l4 = reinterpret_cast<uint4 *>(lds);
        const int n16 = copies > 1 ? copies * copy_stride / 16 : lds_n / 2;
        for (int t = threadIdx.x; t < n16; t += blockDim.x) l4[t] = make_uint4(0u, 0u, 0u, 0u);
    }
    if (stamp) tl[(size_t)blockIdx.x * kTimelineStamps + 6] = (unsigned long long)wall_clock64();
    if (pwave) parent_cut(ks, lane, d, s_cf, s_cc, eflag);
    lds_barrier();
    // workgroup 0 records the parents' cuts in the model (the gains after the adds)
    const bool rec = pwave && blockIdx.x == 0 && rec_f;
    const double rg = rec ? record_parent_cut(s_cf, s_cc, lane, d, cslices, cand_gain, rec_f,
                                              rec_c) : 0.0;
    const unsigned long long t_table = stamp ? (unsigned long long)wall_clock64() : 0ull;
    unsigned long long t_first = 0ull;
    uint32_t cut[4] = {0u, 0u, 0u, 0u};
    if (ROUTED && NP > 0 && layer >= 1) {
#pragma unroll
        for (int kk = 0; kk < (NP > 0 ? NP : 1); ++kk) cut[kk] = s_cc[kk];
    }

    // two steps in flight: the loads of step s + 1 are issued before the
    // adds of step s.  They are issued unconditionally (the last step
    // reloads its own events) so that the waits for step s never cover them.
    if (ia < end) {
        hist_load_rows<ROUTED, NP, FPG, SIGNED, MISS>(A, a, s_cf, ia);
        for (;;) {
            const int64_t ib = ia + stride;
            const bool more_b = ib < end;
            hist_load<ROUTED, NP, FPG, SIGNED, MISS>(B, a, s_cf, more_b ? ib : ia, true);
            hist_add<ROUTED, NP, FPG, SIGNED, MISS>(A, a, lds_lane, writer, s_cf, s_cc, cut, ia, eflag);
            if (stamp && t_first == 0ull) t_first = (unsigned long long)wall_clock64();
            if (!more_b) break;
            ia = ib + stride;
            const bool more_a = ia < end;
            hist_load<ROUTED, NP, FPG, SIGNED, MISS>(A, a, s_cf, more_a ? ia : ib, true);
            hist_add<ROUTED, NP, FPG, SIGNED, MISS>(B, a, lds_lane, writer, s_cf, s_cc, cut, ib, eflag);
            if (!more_a) break;
        }
    }
    lds_barrier();
    if (rec) rec_g[lane] = rg;
    const unsigned long long t_adds = stamp ? (unsigned long long)wall_clock64() : 0ull;
    hist_write_rows(lds, copies, copy_stride, lds_n, a.nk, a.nf, FPG, a.k0, a.j0, a.jstep, d,
                    nbins, a.miss, prefix,
                    reinterpret_cast<uint4 *>(partial + (size_t)p * hnodes * d * nbins * 2), eflag);
    if (eflag) atomicOr(err, eflag);
    if (stamp) {
        unsigned long long *row = tl + (size_t)blockIdx.x * kTimelineStamps;
        row[0] = t_entry;
        row[1] = t_table;
        row[2] = t_first;
        row[3] = t_adds;
        row[4] = (unsigned long long)wall_clock64();
    }
}

// Reference passes of the histogram pass's roofline (measurement only),
// launched with the pass's own grid, workgroup size and dynamic LDS.  kind
// 0: every workgroup returns at once (launch and teardown cost).  kind 1:
// every workgroup reads what the pass reads for its (event chunk, feature
// group), kHistE events per thread and step: the weights, the node ids (if
// any) and the codes of its features, folded into an XOR that is stored only
// if it equals a constant, so that the loads stay and nothing is written.
__global__ __launch_bounds__(1024) void hist_reference_kernel(
    int kind, const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d, int fpg,
    const uint8_t *__restrict__ node, const float *__restrict__ w, int G, int NG, int chunks,
    int64_t chunk_events, int64_t xcd_events, uint32_t *__restrict__ sink) {
    if (kind == 0) return;
    const int groups = G * NG;
    const int cpx = chunks / kXcds;
    const int per_xcd = cpx * groups;   // the grid is kXcds * cpx * groups workgroups
    const int q = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    if (q >= chunks * groups) return;
    const int p = q / groups;
    const int g = (q - p * groups) % G;
    const int64_t xlo = (int64_t)(p / cpx) * xcd_events;
    const int64_t start = xlo + (int64_t)(p % cpx) * chunk_events;
    const int64_t end = min(min(n, xlo + xcd_events), start + chunk_events);
    const int64_t stride = (int64_t)kHistE * blockDim.x;
    uint32_t acc = 0u;
    if (kind == 2 && fpg <= 2) {
        // up to 4 steps per thread, all loads issued before any is used
        uint4 x[4], y[4];
        uint2 nd[4], c0[4], c1[4];
        if (end <= start) return;
        const int64_t i0 = start + (int64_t)kHistE * threadIdx.x;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
            // a whole step inside the chunk's padded range (start is a multiple of 8)
            const int64_t i = min(i0 + k * stride, end - 1) / kHistE * kHistE;
            x[k] = reinterpret_cast<const uint4 *>(w + i)[0];
            y[k] = reinterpret_cast<const uint4 *>(w + i)[1];
            nd[k] = node ? *reinterpret_cast<const uint2 *>(node + i) : make_uint2(0u, 0u);
            c0[k] = *reinterpret_cast<const uint2 *>(xb + (int64_t)min(g, d - 1) * ldb + i);
            c1[k] = *reinterpret_cast<const uint2 *>(xb + (int64_t)min(g + G, d - 1) * ldb + i);
        }
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (i0 + k * stride < end)
                acc ^= x[k].x ^ x[k].y ^ x[k].z ^ x[k].w ^ y[k].x ^ y[k].y ^ y[k].z ^ y[k].w ^
                       nd[k].x ^ nd[k].y ^ c0[k].x ^ c0[k].y ^ c1[k].x ^ c1[k].y;
        if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
        return;
    }
    for (int64_t i = start + (int64_t)kHistE * threadIdx.x; i < end; i += stride) {
        const uint4 x = reinterpret_cast<const uint4 *>(w + i)[0];
        const uint4 y = reinterpret_cast<const uint4 *>(w + i)[1];
        acc ^= x.x ^ x.y ^ x.z ^ x.w ^ y.x ^ y.y ^ y.z ^ y.w;
        if (node) {
            const uint2 nd = *reinterpret_cast<const uint2 *>(node + i);
            acc ^= nd.x ^ nd.y;
        }
        for (int ff = 0; ff < fpg; ++ff) {
            const uint2 c = *reinterpret_cast<const uint2 *>(
                xb + (int64_t)min(g + ff * G, d - 1) * ldb + i);
            acc ^= c.x ^ c.y;
        }
    }
    if (acc == 0x9E3779B9u) sink[blockIdx.x] = acc;
}

// Sum of the fixed-point chunk partials (exact) converted to float64, plus
// the float64 side histogram.
__global__ __launch_bounds__(256) void merge_partials_kernel(const uint64_t *__restrict__ partial,
                                                             int chunks, size_t count, int scale,
                                                             const double *__restrict__ small,
                                                             double *__restrict__ out) {
    for (size_t i = blockIdx.x * (size_t)blockDim.x + threadIdx.x; i < count;
         i += (size_t)gridDim.x * blockDim.x) {
        uint64_t s = 0;
        for (int p = 0; p < chunks; ++p) s += partial[(size_t)p * count + i];
        out[i] = ldexp((double)(long long)s, -scale) + small[i];
    }
}

// Sum of |w| (fixed grid, fixed reduction order): per-block partials, then
// one block adds them.
__global__ __launch_bounds__(256) void abs_sum_kernel(const float *__restrict__ w, int64_t n,
                                                      double *__restrict__ block_partial) {
    double s = 0.0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        s += (double)fabsf(w[i]);
    for (int off = kWave / 2; off > 0; off >>= 1) s += __shfl_down(s, off);
    __shared__ double ws[256 / kWave];
    if (threadIdx.x % kWave == 0) ws[threadIdx.x / kWave] = s;
    __syncthreads();
    if (threadIdx.x == 0) {
        double t = 0.0;
        for (int k = 0; k < (int)(blockDim.x / kWave); ++k) t += ws[k];
        block_partial[blockIdx.x] = t;
    }
}

__global__ void sum_blocks_kernel(const double *__restrict__ block_partial, int nblocks,
                                  double *__restrict__ out) {
    if (threadIdx.x == 0 && blockIdx.x == 0) {
        double t = 0.0;
        for (int k = 0; k < nblocks; ++k) t += block_partial[k];
        *out = t;
    }
}

// ---------------------------------------------------------------------------
// Best cut of every (node, feature) of a float64 histogram (the standalone
// step): one wavefront per (node, feature); lane l owns bins 4l..4l+3, builds
// the cumulative histograms with an in-lane prefix plus a wavefront scan,
// evaluates the separation gain of each candidate cut and reduces to the best
// (gain highest, then lowest bin) as entry [node][feature] of a candidate set
// with one slice per feature.
//
// Exactness rules shared with the plain definition: a cut whose left or
// right side holds no event has gain exactly 0 (as the definition gives
// with exact zero sums); a cut c >= 2 whose bin c-1 is empty makes the same
// partition as cut c-1, has the same gain in exact arithmetic, and is
// skipped so that the lower cut wins the tie independently of rounding.
__global__ __launch_bounds__(kWave) void best_cuts_f64_kernel(const double *__restrict__ hist,
                                                              int d, int nbins,
                                                              double *__restrict__ cand_gain,
                                                              int *__restrict__ cand_cut) {
#pragma clang fp contract(off)
    const int lane = threadIdx.x;
    const int pair = blockIdx.x;   // node * d + feature
    const int b0 = 4 * lane;
    const int nb = b0 < nbins ? min(4, nbins - b0) : 0;
    const size_t off = (size_t)pair * nbins * 2 + 2 * b0;
    double hs[4] = {0.0, 0.0, 0.0, 0.0}, hb[4] = {0.0, 0.0, 0.0, 0.0};
    for (int e = 0; e < nb; ++e) {
        hs[e] = hist[off + 2 * e];
        hb[e] = hist[off + 2 * e + 1];
    }
    bool ne[4];
    int first = 0x7fffffff, last = -1;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        ne[e] = (hs[e] != 0.0) || (hb[e] != 0.0);
        if (ne[e]) {
            first = min(first, b0 + e);
            last = max(last, b0 + e);
        }
    }
    double ps[4], pb[4];   // in-lane inclusive prefix
    ps[0] = hs[0];
    pb[0] = hb[0];
#pragma unroll
    for (int e = 1; e < 4; ++e) {
        ps[e] = ps[e - 1] + hs[e];
        pb[e] = pb[e - 1] + hb[e];
    }
    double is = ps[3], ib = pb[3];   // wavefront inclusive scan of the lane totals
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
        const double us = __shfl_up(is, o);
        const double ub = __shfl_up(ib, o);
        if (lane >= o) {
            is += us;
            ib += ub;
        }
    }
    double xs = __shfl_up(is, 1), xbk = __shfl_up(ib, 1);
    if (lane == 0) {
        xs = 0.0;
        xbk = 0.0;
    }
    const double ST = __shfl(is, kWave - 1);
    const double BT = __shfl(ib, kWave - 1);
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        first = min(first, __shfl_xor(first, o));
        last = max(last, __shfl_xor(last, o));
    }
    const bool prev_ne = __shfl_up(ne[3] ? 1 : 0, 1) != 0;
    const double gp = gini(ST, BT);
    double best = -INFINITY;
    int bestc = 0x7fffffff;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const int c = b0 + e;
        if (c < 1 || c > nbins - 1) continue;
        const bool below_ne = e > 0 ? ne[e - 1] : prev_ne;
        if (c >= 2 && !below_ne) continue;
        double g;
        if (c <= first || c > last) {
            g = 0.0;
        } else {
            const double S = e > 0 ? xs + ps[e - 1] : xs;
            const double B = e > 0 ? xbk + pb[e - 1] : xbk;
            g = (gp - gini(S, B)) - gini(ST - S, BT - B);
        }
        if (g > best) {
            best = g;
            bestc = c;
        }
    }
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const double og = __shfl_xor(best, o);
        const int oc = __shfl_xor(bestc, o);
        if (og > best || (og == best && oc < bestc)) {
            best = og;
            bestc = oc;
        }
    }
    if (lane == 0) {
        cand_gain[pair] = best;
        cand_cut[pair] = bestc;
    }
}

// ---------------------------------------------------------------------------
// Best cuts of a layer in the fit (cumulative histograms, separation gain,
// argmax; section 1.1), from the prefix-summed fixed-point chunk partials of
// the routed histogram pass: summed over chunks, the partial row of a
// (node, feature) is P(b) = the node's histogram summed over bins <= b, per
// class, exactly (64-bit integers).  Cut c (1 <= c <= B-1) sends bins < c
// left, so S(c) = P_sig(c-1) and B(c) = P_bkg(c-1); the totals are P(B-1).
//
// The cuts of a row are split into slices of kCutSlice cuts, one workgroup
// per (histogrammed node, feature, slice): slice q holds cuts
// kCutSlice q + 1 .. kCutSlice (q + 1) and needs P at bins
// kCutSlice q - 1 .. kCutSlice q + kCutSlice - 1 (P(c-1) of its cuts and, for
// the empty-bin rule, P(c-2)): lane l holds window bin l >> 1, class l & 1.
// The workgroup's wavefronts sum the chunks round-robin (integer sums: exact
// in any order); wavefront 0 then evaluates the slice's cuts and writes the
// slice's candidate (entry j * S + q of the node, gain highest, then lowest
// bin).  Below the root (kCutSibling) a workgroup takes a parent: the
// partials are one child of each parent (the left one, or as the list pass
// flags it the right one), wavefronts 0 and 1 evaluate the left and right
// children, and the other child is formed as parent - child from the
// parents' summed rows (hparent).  With missing values (kCutStopped, section
// 4.2) the events that stopped at the parent have partials of their own and
// the other child is parent - child - stopped.  hout receives the summed
// rows of every node of the layer (the next layer's parents).
//
// The side histogram (float64 sums of the weights below the fixed-point
// grid, per node of the layer, plain bins) is added after a prefix scan when
// any of a row's values is non-zero.  Every workgroup also clears its share
// of the next layer's side histogram (small_next), which no kernel reads in
// the meantime.
//
// Exactness rules (those of the plain definition, decided here on the exact
// sums): a cut with an empty side has gain exactly 0; a cut c >= 2 whose bin
// c-1 is empty makes the same partition as cut c-1 and is skipped, so the
// lower cut wins that tie whatever the rounding.
constexpr int kCutWaves = 4;

template <int MODE>   // CutMode
__global__ __launch_bounds__(kCutWaves * kWave) void cut_scan_kernel(
    const uint64_t *__restrict__ partial, int chunks, int scale, const double *__restrict__ small,
    double *__restrict__ small_next, size_t small_next_count, int hnodes, int d, int nbins, int S,
    double *__restrict__ cand_gain, int *__restrict__ cand_cut,
    const uint64_t *__restrict__ hparent, uint64_t *__restrict__ hout,
    const uint2 *__restrict__ lchunks, uint32_t *__restrict__ clear_words, int clear_count,
    const uint32_t *__restrict__ sany, uint32_t *__restrict__ sany_next,
    unsigned long long *__restrict__ keys, unsigned long long *__restrict__ keys_next) {
#pragma clang fp contract(off)
    constexpr bool PAIR = MODE != kCutPlain;   // both children of a parent per workgroup
    __shared__ uint64_t red[kCutWaves][kWave + 2];
    __shared__ uint64_t red_stop[MODE == kCutStopped ? kCutWaves : 1][kWave + 2];
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    // row kj = (node or parent, feature) and slice q.  The S slices of a row
    // run on one XCD (workgroup b runs on XCD b % 8), so that the cache
    // lines that adjacent slices' windows share, and the row totals that
    // every slice reads, come from that XCD's L2; the grid is padded to
    // whole rounds of 8 rows
    const int rows = (MODE == kCutStopped ? hnodes / 2 : hnodes) * d;
    const int xq = blockIdx.x % kXcds, pq = blockIdx.x / kXcds;
    const int q = pq % S;
    const int kj0 = (pq / S) * kXcds + xq;
    const bool valid = kj0 < rows;
    const int kj = valid ? kj0 : 0;
    const int j = kj % d;
    const int k = kj / d;   // histogrammed node, or with PAIR the parent
    const size_t row = (size_t)nbins * 2;
    const int wi = lane >> 1, cls = lane & 1;
    const int b = kCutSlice * q - 1 + wi;   // this lane's window bin
    const bool inb = b >= 0 && b < nbins;
    // slots: the histogrammed child (or node) and, with kCutStopped, the
    // events that stopped at the parent.  Partials of the streaming pass:
    // [chunks][hnodes][d][B][2]; of the list pass (lchunks): chunk c of slot
    // s at [base_s + c][d][B][2], and the flag of a child slot tells that it
    // holds the right child
    const int cslot = MODE == kCutStopped ? 2 * k : k;
    uint32_t cbase = (uint32_t)cslot, sbase = (uint32_t)cslot + 1u, flag = 0u;
    int cchunks = valid ? chunks : 0, schunks = valid && MODE == kCutStopped ? chunks : 0;
    if (lchunks && valid) {
        const uint2 lc = lchunks[cslot];
        cbase = lc.x;
        cchunks = (int)(lc.y & 0x7fffffffu);
        flag = lc.y >> 31;
        if (MODE == kCutStopped) {
            const uint2 ls = lchunks[cslot + 1];
            sbase = ls.x;
            schunks = (int)(ls.y & 0x7fffffffu);
        }
    }
    // offsets of this lane's window bin and of the row total within a row
    // [k][j] of the parents' rows, and within the first chunk's partial rows
    const size_t off = ((size_t)k * d + j) * row;
    const size_t wv = (size_t)(inb ? b : 0) * 2 + cls, wt = (size_t)(nbins - 1) * 2 + cls;
    const size_t coff = ((size_t)cbase * d + j) * row, soff = ((size_t)sbase * d + j) * row;
    const size_t stride_p = lchunks ? (size_t)d * row : (size_t)hnodes * d * row;
    // node of this wavefront's candidates, as an index within the layer; with
    // PAIR wavefront `sub` forms its node as parent - the histogrammed child
    // (- the stopped events)
    const int node = PAIR ? 2 * k + (wave & 1) : k;
    const int sub = flag ? 0 : 1;
    const size_t noff = ((size_t)node * d + j) * row;

    // side histogram row of the candidate wavefronts' node: lane l holds bins
    // 4l..4l+3, both classes.  Without sany it is loaded first, in flight
    // with the chunk sums; with sany (list layers, where the nine slices of
    // a row would each read all of it and the row is nearly always empty)
    // only after them, and only if *sany says a weight went to the layer's
    // side histogram
    double sd[8];
    const bool cwave = wave < (PAIR ? 2 : 1);
    auto side_load = [&]() {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int bb = 4 * lane + (e >> 1);
            sd[e] = bb < nbins ? small[noff + 2 * bb + (e & 1)] : 0.0;
        }
    };
#pragma unroll
    for (int e = 0; e < 8; ++e) sd[e] = 0.0;
    if (cwave && valid && !sany) side_load();
    uint64_t pv = 0, pt = 0;   // parent row (other child = parent - histogrammed child)
    if (PAIR && wave == sub) {
        pv = hparent[off + wv];
        pt = hparent[off + wt];
    }
    // chunk sums: wavefront w takes chunks w, w + kCutWaves, ...
    auto chunk_sums = [&](size_t base_off, int nch, uint64_t &v, uint64_t &vt) {
        const size_t ov = base_off + wv, ot = base_off + wt;
        int p = wave;
        for (; p + 3 * kCutWaves < nch; p += 4 * kCutWaves) {
            const uint64_t *b0 = partial + (size_t)p * stride_p;
            const uint64_t *b1 = b0 + kCutWaves * stride_p;
            const uint64_t *b2 = b1 + kCutWaves * stride_p;
            const uint64_t *b3 = b2 + kCutWaves * stride_p;
            const uint64_t x0 = b0[ov], x1 = b1[ov], x2 = b2[ov], x3 = b3[ov];
            const uint64_t t0 = b0[ot], t1 = b1[ot], t2 = b2[ot], t3 = b3[ot];
            v += (x0 + x1) + (x2 + x3);
            vt += (t0 + t1) + (t2 + t3);
        }
        for (; p < nch; p += kCutWaves) {
            v += partial[(size_t)p * stride_p + ov];
            vt += partial[(size_t)p * stride_p + ot];
        }
    };
    uint64_t v = 0, vt = 0;
    chunk_sums(coff, cchunks, v, vt);
    red[wave][lane] = v;
    if (lane < 2) red[wave][kWave + lane] = vt;
    if (cwave && valid && sany && *sany != 0u) side_load();
    if (MODE == kCutStopped) {
        uint64_t sv = 0, st = 0;
        chunk_sums(soff, schunks, sv, st);
        red_stop[wave][lane] = sv;
        if (lane < 2) red_stop[wave][kWave + lane] = st;
    }
    // this workgroup's share of the next layer's side histogram; workgroup
    // 0 also clears clear_words (counters of the next passes)
    {
        const size_t per = (small_next_count + gridDim.x - 1) / gridDim.x;
        const size_t lo = per * blockIdx.x;
        const size_t hi = min(small_next_count, lo + per);
        for (size_t t = lo + threadIdx.x; t < hi; t += blockDim.x) small_next[t] = 0.0;
        if (sany_next && blockIdx.x == 0 && threadIdx.x == 0) *sany_next = 0u;
        if (keys_next && blockIdx.x == 0)
            for (int t = threadIdx.x; t < kKeyNodes * kXcds; t += blockDim.x)
                keys_next[(size_t)t * kKeyStride] = 0ull;
        if (clear_words && blockIdx.x == 0)
            for (int t = threadIdx.x; t < clear_count; t += blockDim.x) clear_words[t] = 0u;
    }
    lds_barrier();
    if (!cwave || !valid) return;
    uint64_t P = 0, T = 0;
#pragma unroll
    for (int w = 0; w < kCutWaves; ++w) {
        P += red[w][lane];
        T += red[w][kWave + cls];
    }
    if (PAIR && wave == sub) {   // the other child = parent - histogrammed child (exact)
        P = pv - P;
        T = pt - T;
        if (MODE == kCutStopped) {   // - the events that stopped at the parent (exact)
#pragma unroll
            for (int w = 0; w < kCutWaves; ++w) {
                P -= red_stop[w][lane];
                T -= red_stop[w][kWave + cls];
            }
        }
    }
    if (!inb) P = 0;
    if (hout && wi >= 1 && inb) hout[noff + 2 * b + cls] = P;
    // the row total P(B-1), which the windows do not reach when B > 31 S
    if (hout && q == S - 1 && lane < 2) hout[noff + 2 * (nbins - 1) + cls] = T;

    // side histogram: inclusive prefix over bins (per class) when the row
    // holds anything, picked at this lane's window bin; sb = the bin itself
    double sp = 0.0, sb = 0.0, stot = 0.0;
    bool any = false;
    int side_last = -1;   // highest bin with side weight (either class), exact
#pragma unroll
    for (int e = 0; e < 8; ++e) {
        any |= sd[e] != 0.0;
        if (sd[e] != 0.0) side_last = max(side_last, 4 * lane + (e >> 1));
    }
    if (__any(any)) {
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) side_last = max(side_last, __shfl_xor(side_last, o));
        double pr[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) pr[e] = sd[e] + (e >= 2 ? pr[e - 2] : 0.0);
        double xs = pr[6], xb = pr[7];   // lane totals, inclusive scan
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const double us = __shfl_up(xs, o), ub = __shfl_up(xb, o);
            if (lane >= o) {
                xs += us;
                xb += ub;
            }
        }
        const double es = xs - pr[6], eb = xb - pr[7];   // exclusive
        const int src = inb ? b >> 2 : 0, el = inb ? b & 3 : 0;
        double cand_p = 0.0, cand_b = 0.0;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const double ps = __shfl(pr[2 * e] + es, src), pbk = __shfl(pr[2 * e + 1] + eb, src);
            const double vs = __shfl(sd[2 * e], src), vb = __shfl(sd[2 * e + 1], src);
            if (el == e) {
                cand_p = cls ? pbk : ps;
                cand_b = cls ? vb : vs;
            }
        }
        sp = inb ? cand_p : 0.0;
        sb = inb ? cand_b : 0.0;
        const double tS = __shfl(xs, kWave - 1), tB = __shfl(xb, kWave - 1);
        stot = cls ? tB : tS;
    }

    // cut c = kCutSlice q + wi evaluated by the even lane of pair wi >= 1:
    // this pair holds bin c-1, the pair below bin c-2
    const unsigned long long Ps = __shfl((unsigned long long)P, lane & ~1);
    const unsigned long long Pb = __shfl((unsigned long long)P, lane | 1);
    const unsigned long long Qs = __shfl((unsigned long long)P, max((lane & ~1) - 2, 0));
    const unsigned long long Qb = __shfl((unsigned long long)P, max((lane & ~1) - 1, 1));
    const unsigned long long Ts = __shfl((unsigned long long)T, 0);
    const unsigned long long Tb = __shfl((unsigned long long)T, 1);
    const double sPs = __shfl(sp, lane & ~1), sPb = __shfl(sp, lane | 1);
    const double sBs = __shfl(sb, lane & ~1), sBb = __shfl(sb, lane | 1);
    const double sTs = __shfl(stot, 0), sTb = __shfl(stot, 1);
    const int c = kCutSlice * q + wi;
    double g = -INFINITY;
    if (cls == 0 && wi >= 1 && c <= nbins - 1) {
        // empty sides from exact quantities: the fixed-point sums, and for the
        // side histogram a zero prefix below c, or no weight in a bin at or
        // above c (side_last)
        const bool left_empty = Ps == 0 && Pb == 0 && sPs == 0.0 && sPb == 0.0;
        const bool right_empty = Ps == Ts && Pb == Tb && c > side_last;
        const bool bin_empty = Ps == Qs && Pb == Qb && sBs == 0.0 && sBb == 0.0;
        if (c >= 2 && bin_empty) {
            g = -INFINITY;   // same partition as cut c-1
        } else if (left_empty || right_empty) {
            g = 0.0;
        } else {
            // fixed-point sums as signed integers (negative event weights)
            const double SS = ldexp((double)(long long)Ps, -scale) + sPs;
            const double BB = ldexp((double)(long long)Pb, -scale) + sPb;
            const double ST = ldexp((double)(long long)Ts, -scale) + sTs;
            const double BT = ldexp((double)(long long)Tb, -scale) + sTb;
            g = (gini(ST, BT) - gini(SS, BB)) - gini(ST - SS, BT - BB);
        }
    }
    double best = g;
    int bestc = g > -INFINITY ? c : 0x7fffffff;
#pragma unroll
    for (int o = kWave / 2; o > 0; o >>= 1) {
        const double og = __shfl_xor(best, o);
        const int oc = __shfl_xor(bestc, o);
        if (og > best || (og == best && oc < bestc)) {
            best = og;
            bestc = oc;
        }
    }
    if (lane == 0) {
        const size_t e = (size_t)node * d * S + (size_t)j * S + q;
        cand_gain[e] = best;
        cand_cut[e] = bestc;
        if (keys && best > -INFINITY)   // the slot of this workgroup's XCD
            atomicMax(keys + ((size_t)node * kXcds + xq) * kKeyStride, cut_key(best, j, bestc));
    }
}

// ---------------------------------------------------------------------------
// Terminal boost weights (section 1.3): per leaf, sum(v y~) and
// sum(v |y~| (2 - |y~|)) over the sampled events, one partial per
// workgroup, from yts (y~ of the sampled events, 0 for the others, written
// by the re-weighting pass).  Routed mode first takes the last layer's cuts
// from their best-cut keys, sends every event from layer depth-1 to its leaf
// and stores the leaf id; with at most four parents the code rows of the
// parents' cut features are loaded with the step's other data, so routing
// costs no dependent load.
//
// Every column of the LDS array acc[value][column] holds the 2 * slots
// accumulators of `share` consecutive threads, which add their events in
// turn (non-returning LDS float64 adds: each address has one writer at a
// time, in a fixed order, and no bank conflicts); the workgroup then adds
// its columns in a fixed order.  The columns take up to ~130 KiB, so deep
// trees have few of them: up to 8 threads share one there, which keeps 512
// threads (8 wavefronts) per CU instead of 128 or 64.
// kLeafE consecutive events per thread and step on padded arrays (weights,
// yts, node ids: zero pseudo-response beyond n), the next step's loads
// issued before the current step's arithmetic.
constexpr int kLeafE = 8;

// Terminal-node slots of the leaf pass: the 2^D leaves, or with missing
// values every node of the tree (2^(D+1) - 1).
__host__ __device__ constexpr int leaf_slots(int depth, bool missing) {
    return missing ? (2 << depth) - 1 : 1 << depth;
}

__host__ __device__ constexpr int leaf_columns(int depth, bool missing) {
    // acc takes columns * 2 slots doubles: at most ~136 KiB (depth 7 with
    // missing values: 255 slots in 32 columns)
    return 2 * leaf_slots(depth, missing) <= 64    ? 256
           : 2 * leaf_slots(depth, missing) <= 128 ? 128
           : 2 * leaf_slots(depth, missing) <= 256 ? 64
                                                    : 32;
}

// threads per accumulator column
__host__ __device__ constexpr int leaf_share(int depth, bool missing) {
    return leaf_columns(depth, missing) >= 256 ? 1 : 512 / leaf_columns(depth, missing);
}

__host__ __device__ constexpr int leaf_threads(int depth, bool missing) {
    return leaf_columns(depth, missing) * leaf_share(depth, missing);
}

template <int NP>
struct LeafStep {
    uint2 node;                     // parent ids (routed) or leaf ids
    uint2 rows[NP > 0 ? NP : 1];    // codes of the parents' cut features
    double yt[kLeafE];
    float v[kLeafE];
};

template <bool ROUTED, int NP>
__device__ __forceinline__ void leaf_load_rows(LeafStep<NP> &st, const uint8_t *__restrict__ xb,
                                               int64_t ldb, int d, const uint8_t *s_cf,
                                               int64_t i0) {
    if (ROUTED && NP > 0) {
#pragma unroll
        for (int k = 0; k < (NP > 0 ? NP : 1); ++k)
            st.rows[k] =
                *reinterpret_cast<const uint2 *>(xb + (int64_t)min((int)s_cf[k], d - 1) * ldb + i0);
    }
}

template <bool ROUTED, int NP>
__device__ __forceinline__ void leaf_load(LeafStep<NP> &st, const uint8_t *__restrict__ xb,
                                          int64_t ldb, int d, const uint8_t *__restrict__ node_in,
                                          const float *__restrict__ v,
                                          const double *__restrict__ yts, const uint8_t *s_cf,
                                          int64_t i0, bool with_rows) {
    st.node = node_in ? *reinterpret_cast<const uint2 *>(node_in + i0)
                      : make_uint2(0x01010101u, 0x01010101u);
#pragma unroll
    for (int e = 0; e < kLeafE; e += 2) {
        const double2 y2 = *reinterpret_cast<const double2 *>(yts + i0 + e);
        st.yt[e] = y2.x;
        st.yt[e + 1] = y2.y;
    }
    if (v) {
        const float4 a = reinterpret_cast<const float4 *>(v + i0)[0];
        const float4 b = reinterpret_cast<const float4 *>(v + i0)[1];
        st.v[0] = a.x; st.v[1] = a.y; st.v[2] = a.z; st.v[3] = a.w;
        st.v[4] = b.x; st.v[5] = b.y; st.v[6] = b.z; st.v[7] = b.w;
    } else {
#pragma unroll
        for (int e = 0; e < kLeafE; ++e) st.v[e] = 1.0f;
    }
    if (with_rows) leaf_load_rows<ROUTED, NP>(st, xb, ldb, d, s_cf, i0);
}

template <bool ROUTED, int NP>
__global__ __launch_bounds__(512) void leaf_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d,
    const uint8_t *__restrict__ node_in, uint8_t *__restrict__ node_out,
    const double *__restrict__ cand_gain, const unsigned long long *__restrict__ keys, int cslices,
    uint8_t *__restrict__ rec_f, uint8_t *__restrict__ rec_c, double *__restrict__ rec_g,
    int depth, bool missing, const float *__restrict__ v, const double *__restrict__ yts,
    double *__restrict__ leaf_partial, int *__restrict__ err, int64_t xcd_events) {
#pragma clang fp contract(off)
    // Sums per terminal node: the leaves, and with missing values (section
    // 4.2) every node, since an event stops at the node that cuts on its
    // missing value; slot = heap id - first_id.
    extern __shared__ double acc[];   // [2 nslots][ncol + 1], then the segment sums
    __shared__ uint8_t s_cf[64], s_cc[64];
    const int T = blockDim.x;
    const int share = leaf_share(depth, missing);   // threads per column
    const int ncol = T / share;
    const int sub = threadIdx.x & (share - 1);
    const int nleaf = 1 << depth;
    const uint32_t first_id = missing ? 1u : (uint32_t)nleaf;
    const int nslots = missing ? 2 * nleaf - 1 : nleaf;
    const int nv = 2 * nslots;
    const int half = nleaf >> 1;
    const int lane = threadIdx.x % kWave;
    const int wave = threadIdx.x / kWave;
    int eflag = 0;
    // the workgroups on XCD x = blockIdx % 8 take the events [x R, (x + 1) R)
    const int64_t xlo = (int64_t)(blockIdx.x % kXcds) * xcd_events;
    const int64_t xend = min(n, xlo + xcd_events);
    const int64_t stride = (int64_t)(gridDim.x / kXcds) * T * kLeafE;
    int64_t ia = xlo + ((int64_t)(blockIdx.x / kXcds) * T + threadIdx.x) * kLeafE;

    // the parents' best-cut keys (lane k of wavefront 0 takes parent k) in
    // flight with the first step's data
    const bool pwave = ROUTED && wave == 0 && lane < half;
    KeySlots ks;
    if (pwave) key_load(keys, lane, ks);
    LeafStep<NP> A, B;
    if (ia < xend) leaf_load<ROUTED, NP>(A, xb, ldb, d, node_in, v, yts, s_cf, ia, false);
    const int TP = ncol + 1;   // row stride: rows start two LDS banks apart
    for (int t = threadIdx.x; t < nv * TP; t += T) acc[t] = 0.0;
    if (pwave) parent_cut(ks, lane, d, s_cf, s_cc, eflag);
    lds_barrier();
    // workgroup 0 records the parents' cuts in the model (the gains at the end)
    const bool rec = pwave && blockIdx.x == 0 && rec_f;
    const double rg = rec ? record_parent_cut(s_cf, s_cc, lane, d, cslices, cand_gain, rec_f,
                                              rec_c) : 0.0;
    uint32_t cut[4] = {0u, 0u, 0u, 0u};
    if (ROUTED && NP > 0) {
#pragma unroll
        for (int k = 0; k < (NP > 0 ? NP : 1); ++k) cut[k] = s_cc[k];
    }
    double *mine = acc + threadIdx.x / share;   // this thread's column, value stride TP

    auto add = [&](const LeafStep<NP> &st, int64_t i0) {
        uint32_t o[2] = {0u, 0u};
        uint32_t lid[kLeafE];
#pragma unroll
        for (int e = 0; e < kLeafE; ++e) {
            uint32_t leaf;
            if (ROUTED) {
                uint32_t par = byte8(st.node, e);
                uint32_t k = par - (uint32_t)half;
                bool stop = false;
                if (k >= (uint32_t)half) {
                    // below the layer: stopped earlier at a missing value;
                    // above it: unreachable for ids written by this library
                    const bool earlier = missing & (par < (uint32_t)half);
                    stop = earlier;
                    if (!earlier) eflag |= kErrRoute;
                    k = 0u;
                    par = earlier ? par : (uint32_t)half;
                }
                uint32_t x, c;
                if (NP > 0) {
                    x = byte8(st.rows[0], e);
                    c = cut[0];
#pragma unroll
                    for (int kk = 1; kk < (NP > 0 ? NP : 1); ++kk) {
                        if (k == (uint32_t)kk) {
                            x = byte8(st.rows[kk], e);
                            c = cut[kk];
                        }
                    }
                } else {
                    x = xb[(int64_t)min((int)s_cf[k], d - 1) * ldb + i0 + e];
                    c = s_cc[k];
                }
                stop |= missing & (x == (uint32_t)kMissingCode);
                leaf = stop ? par : 2u * par + (x >= c ? 1u : 0u);
                o[e >> 2] |= leaf << (8 * (e & 3));
            } else {
                leaf = byte8(st.node, e);
            }
            lid[e] = leaf - first_id;
            // unreachable for ids written by this library
            if (st.yt[e] != 0.0 && lid[e] >= (uint32_t)nslots) eflag |= kErrRoute;
        }
        // padded events get leaf ids too (the arrays hold whole steps)
        if (ROUTED) *reinterpret_cast<uint2 *>(node_out + i0) = make_uint2(o[0], o[1]);
        // the threads of a column add their sampled events in turn
        for (int r = 0; r < share; ++r) {
            if (sub == r) {
#pragma unroll
                for (int e = 0; e < kLeafE; ++e) {
                    const double yt = st.yt[e];
                    const uint32_t li = lid[e];
                    if (yt != 0.0 && li < (uint32_t)nslots) {   // sampled
                        const double vi = (double)st.v[e];
                        const double a = fabs(yt);
                        unsafeAtomicAdd(mine + (size_t)(2 * li) * TP, vi * yt);
                        unsafeAtomicAdd(mine + (size_t)(2 * li + 1) * TP, vi * a * (2.0 - a));
                    }
                }
            }
        }
    };
    if (ia < xend) {
        leaf_load_rows<ROUTED, NP>(A, xb, ldb, d, s_cf, ia);
        for (;;) {
            const int64_t ib = ia + stride;
            const bool more_b = ib < xend;
            leaf_load<ROUTED, NP>(B, xb, ldb, d, node_in, v, yts, s_cf, more_b ? ib : ia, true);
            add(A, ia);
            if (!more_b) break;
            ia = ib + stride;
            const bool more_a = ia < xend;
            leaf_load<ROUTED, NP>(A, xb, ldb, d, node_in, v, yts, s_cf, more_a ? ia : ib, true);
            add(B, ib);
            if (!more_a) break;
        }
    }
    lds_barrier();
    if (rec) rec_g[lane] = rg;
    // columns added in a fixed order: G segments of T / G columns per value,
    // then the G segment sums; G is a power of two (nv need not be one, so
    // T / nv may not divide T) with G nv <= T
    int G = 1;
    while (2 * G * nv <= ncol) G *= 2;
    const int seg = ncol / G;
    double *segsum = acc + (size_t)nv * TP;   // [G][nv]
    for (int idx = threadIdx.x; idx < nv * G; idx += T) {
        const int val = idx % nv, g = idx / nv;
        const double *col = acc + (size_t)val * TP + g * seg;
        double s0 = 0.0, s1 = 0.0;
        for (int c = 0; c < seg; c += 2) {
            s0 += col[c];
            s1 += col[c + 1];
        }
        segsum[g * nv + val] = s0 + s1;
    }
    lds_barrier();
    for (int val = threadIdx.x; val < nv; val += T) {
        double sum = 0.0;
        for (int g = 0; g < G; ++g) sum += segsum[g * nv + val];
        leaf_partial[(size_t)blockIdx.x * nv + val] = sum;
    }
    if (eflag) atomicOr(err, eflag);
}

__global__ __launch_bounds__(kLeafReduceThreads) void leaf_finalize_kernel(
    const double *__restrict__ leaf_partial, int nblocks, int nslots, int inner, double eta,
    double *__restrict__ leaf_out) {
    __shared__ double red[kLeafReduceThreads];
    __shared__ double s_leaf[kLeafSumSlots];
    reduce_leaf_partials(leaf_partial, nblocks, nslots, eta, red, s_leaf, inner);
    for (int t = threadIdx.x; t < nslots; t += blockDim.x) leaf_out[t] = s_leaf[t];
}

// Routing of one layer as a pass of its own, for layers with more parents
// than the histogram pass routes itself.  There each event would gather one
// code byte from the row of its parent's cut feature (a cache line per lane
// of the load, as the parents of a wavefront's events differ), once in every
// feature group's workgroup; here the gather happens once per event.  Every
// workgroup takes the parents' cuts from their best-cut keys (workgroup 0
// records them in the model), then moves each event of its XCD's range to
// its node of this layer, node <- 2 node + [code >= cut] (section 1.1).
// With miss, an event whose code of the cut feature is the missing code, or
// which stopped at an earlier layer, keeps its node (section 4.2).  Whole
// steps of kHistE events: padded events get ids too.
constexpr int kRouteLayerThreads = 1024;
__global__ __launch_bounds__(kRouteLayerThreads) void route_layer_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d,
    const uint8_t *__restrict__ node_in, uint8_t *__restrict__ node_out,
    const double *__restrict__ cand_gain, const unsigned long long *__restrict__ keys, int cslices,
    uint8_t *__restrict__ rec_f, uint8_t *__restrict__ rec_c, double *__restrict__ rec_g,
    int layer, bool miss, int *__restrict__ err, int64_t xcd_events) {
    __shared__ uint8_t s_cf[64], s_cc[64];
    const uint32_t half = 1u << (layer - 1);
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    int eflag = 0;
    // the parents' cuts from their best-cut keys (lane k of wavefront 0 takes parent k)
    const bool pwave = wave == 0 && lane < (int)half;
    if (pwave) {
        KeySlots ks;
        key_load(keys, lane, ks);
        parent_cut(ks, lane, d, s_cf, s_cc, eflag);
    }
    __syncthreads();
    // workgroup 0 records them in the model (the gains at the end)
    const bool rec = pwave && blockIdx.x == 0 && rec_f;
    const double rg = rec ? record_parent_cut(s_cf, s_cc, lane, d, cslices, cand_gain, rec_f,
                                              rec_c) : 0.0;
    // the workgroups on XCD x = blockIdx % 8 take the events [x R, (x + 1) R)
    const int64_t xlo = (int64_t)(blockIdx.x % kXcds) * xcd_events;
    const int64_t xend = min(n, xlo + xcd_events);
    const int64_t stride = (int64_t)(gridDim.x / kXcds) * blockDim.x * kHistE;
    for (int64_t i0 = xlo + ((int64_t)(blockIdx.x / kXcds) * blockDim.x + threadIdx.x) * kHistE;
         i0 < xend; i0 += stride) {
        const uint2 pin = *reinterpret_cast<const uint2 *>(node_in + i0);
        uint32_t par[kHistE], k[kHistE], code[kHistE];
        // the step's gathers first, all in flight together
#pragma unroll
        for (int e = 0; e < kHistE; ++e) {
            par[e] = byte8(pin, e);
            k[e] = par[e] - half;
            const uint32_t kk = k[e] < half ? k[e] : 0u;
            code[e] = xb[(int64_t)min((int)s_cf[kk], d - 1) * ldb + i0 + e];
        }
        uint32_t o[2] = {0u, 0u};
#pragma unroll
        for (int e = 0; e < kHistE; ++e) {
            uint32_t p = par[e], kk = k[e];
            bool stop = false;
            if (kk >= half) {
                // below the layer: stopped earlier at a missing value; above
                // it: unreachable for ids written by this library
                const bool earlier = miss & (p < half);
                stop = earlier;
                if (!earlier) eflag |= kErrRoute;
                kk = 0u;
                p = earlier ? p : half;
            }
            stop |= miss & (code[e] == (uint32_t)kMissingCode);
            const uint32_t ne = stop ? p : 2u * p + (code[e] >= s_cc[kk] ? 1u : 0u);
            o[e >> 2] |= ne << (8 * (e & 3));
        }
        *reinterpret_cast<uint2 *>(node_out + i0) = make_uint2(o[0], o[1]);
    }
    if (rec) rec_g[lane] = rg;
    if (eflag) atomicOr(err, eflag);
}

// ---------------------------------------------------------------------------
// Event lists of the histogrammed nodes (layers >= 1 of large fits).
//
// The streaming pass reads every event once per (feature group, node group)
// workgroup and adds it with a half-empty wavefront when the sub-sample or
// the sibling rule leaves it out.  Below the root the list-driven pass
// instead reads, per histogrammed node ("slot": the left child of each
// parent, or with missing values each child), the list of the sampled
// events that the node's histogram counts, and takes their codes from an
// event-major copy of the code matrix: every LDS add then has all its lanes
// busy, and an event is read once per feature group.

// xr[i * dr + j] = xb[j * ldb + i] for i < n (j >= d: 0), E events per
// workgroup (dr a multiple of 16, <= 256; E a multiple of 4).  A thread reads
// the words of 4 consecutive events in 4 feature rows, transposes the 4 x 4
// bytes in registers and stores one word per event into an LDS tile
// [E][dr / 4 + 1] (the extra word spreads the stores over the banks); the
// tile's rows of events < n are then written out as consecutive words.
constexpr int kTransposeThreads = 256;
__global__ __launch_bounds__(kTransposeThreads) void transpose_codes_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d, uint8_t *__restrict__ xr,
    int dr, int E) {
    extern __shared__ uint32_t tile[];
    const int W = dr / 4, WS = W + 1;
    const int64_t i0 = (int64_t)blockIdx.x * E;
    for (int t = threadIdx.x; t < E / 4; t += blockDim.x) {
        const int64_t ie = i0 + 4 * t;
        // bytes of events >= n within the last word read as 0 (rows are
        // padded to ldb >= round_up(n, 16), so the word is in bounds)
        const uint32_t keep = ie + 4 <= n ? 0xffffffffu
                            : ie < n      ? (1u << (8 * (int)(n - ie))) - 1u
                                          : 0u;
        for (int q = 0; q < W; ++q) {
            uint32_t r[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int j = 4 * q + k;
                r[k] = (j < d && keep) ? *reinterpret_cast<const uint32_t *>(xb + (int64_t)j * ldb + ie) & keep
                                       : 0u;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int sh = 8 * e;
                tile[(4 * t + e) * WS + q] = ((r[0] >> sh) & 0xffu) | (((r[1] >> sh) & 0xffu) << 8) |
                                             (((r[2] >> sh) & 0xffu) << 16) |
                                             (((r[3] >> sh) & 0xffu) << 24);
            }
        }
    }
    __syncthreads();
    const int ev = (int)min((int64_t)E, n - i0);
    uint32_t *dst = reinterpret_cast<uint32_t *>(xr + (size_t)i0 * dr);
    for (int o = threadIdx.x; o < ev * W; o += blockDim.x) {   // ev * W <= 32768 / 4
        const int e = o / W;
        dst[o] = tile[e * WS + (o - e * W)];
    }
}

// Routing of layer `layer` (>= 1) for the list-driven histogram pass.  The
// parents' cuts come from their best-cut keys as in route_layer_kernel, and
// every event (node_in = null at layer 1: all at the root) gets its node of
// this layer, node <- 2 node + [code >= cut] (section 1.1); with miss, an
// event whose code of the cut feature is the missing code, or which stopped
// earlier, keeps its node (section 4.2).  A sampled event that has not
// stopped, whose weight is on the fixed-point grid (|w| >= tau) and whose
// node is listed, is appended to the node's list as {event | negative << 31,
// weight bits}; the other events are counted nowhere (the list pass derives
// the next layer's capacities from the lists).  Listed: with lmode kCutSibling one child of every
// parent, the one whose fixed-point weight in the parent's summed rows
// hparent is smaller (lside[k] = 1: the right child; the histogram pass
// takes it and the cut scan forms the other as parent - child), list k =
// parent k; with kCutStopped that child in list 2k and the events that stop
// at parent k here (on the grid) in list 2k + 1 (the other child is parent -
// child - stopped); with kCutPlain every node of the layer, list k = node k.
// List k is the range [start_k,
// start_k + cap_k) of `list`: cap_k = a bound on the on-grid sampled events
// of its node's parent (cap_prev, or cap_root at layer 1), start_k = the caps of the lists
// below k; workgroup 0 records both (lstart, lcap) and lside.  Each
// workgroup counts its entries per list in LDS and reserves them with one
// atomic add per list on cursor[k], so a list holds its events in no fixed
// order (the
// fixed-point sums do not depend on it).  Sampled weights below the grid go
// to the float64 side histogram `small` [2^layer][d][B][2] here, for either
// child and every feature, as the streaming pass adds them.
constexpr int kRouteListThreads = 1024;
// Steps of kHistE events per thread: three (24,576 events per workgroup, so
// that a 10M-event layer needs one round of two workgroups per CU: 41-46 ->
// 37-42 us per layer on workload 4) where the ranks fit the 64 VGPRs that
// this occupancy allows, two otherwise (more live registers: the sign bits
// of signed weights, or 64-bit gather addresses).  OFF32: the code matrix
// spans less than 4 GiB (d * ldb < 2^32), so the gathers take 32-bit
// offsets from its base.
template <bool SIGNED, bool OFF32>
constexpr int route_list_steps() { return OFF32 && !SIGNED ? 3 : 2; }
template <bool SIGNED, bool OFF32>
constexpr int route_list_events() {
    return kRouteListThreads * route_list_steps<SIGNED, OFF32>() * kHistE;
}
template <bool SIGNED, bool OFF32>
__global__ __launch_bounds__(kRouteListThreads, 2 * kRouteListThreads / kWave / 4) void route_list_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d, int nbins,
    const uint8_t *__restrict__ node_in, uint8_t *__restrict__ node_out,
    const float *__restrict__ w, const uint8_t *__restrict__ vsign,
    const double *__restrict__ cand_gain, const unsigned long long *__restrict__ keys, int cslices,
    uint8_t *__restrict__ rec_f, uint8_t *__restrict__ rec_c, double *__restrict__ rec_g,
    int layer, bool miss, int lmode, const uint64_t *__restrict__ hparent, uint32_t tau_bits,
    const uint32_t *__restrict__ cap_prev, uint32_t cap_root,
    uint32_t *__restrict__ cursor, uint32_t *__restrict__ lstart, uint32_t *__restrict__ lcap,
    uint32_t *__restrict__ lside, uint2 *__restrict__ list, double *__restrict__ small,
    int *__restrict__ err, int64_t xcd_events, uint32_t *__restrict__ sany) {
    __shared__ uint8_t s_cf[64], s_cc[64], s_side[64];
    __shared__ uint32_t s_cnt[kListMaxSlots];
    __shared__ uint32_t s_start[kListMaxSlots], s_cap[kListMaxSlots], s_base[kListMaxSlots];
    const uint32_t half = 1u << (layer - 1), nodes = 1u << layer;
    const bool sib = lmode == kCutSibling, stops = lmode == kCutStopped;
    const bool pick = sib || stops;   // one child of each parent listed
    const int nslots = sib ? (int)half : (int)nodes;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int nwaves = blockDim.x / kWave;
    int eflag = 0;
    // the parents' cuts from their best-cut keys (lane k of wavefront 0 takes
    // parent k), and the child listed for each
    const bool pwave = wave == 0 && lane < (int)half;
    if (pwave) {
        const int k = lane;
        int bf, bc;
        bool ok;
        KeySlots ks;
        key_load(keys, k, ks);
        key_cut(key_max(ks), d, &bf, &bc, &ok);
        s_cf[k] = (uint8_t)bf;
        s_cc[k] = (uint8_t)bc;
        if (!ok) eflag |= kErrRoute;
        uint32_t side = 0u;
        if (pick) {
            // weights (signal + background, fixed point) left of the cut
            // and in all, from the parent's prefix-summed row of its feature
            const uint64_t *row = hparent + ((size_t)k * d + bf) * nbins * 2;
            const int64_t left = (int64_t)(row[2 * (bc - 1)] + row[2 * (bc - 1) + 1]);
            const int64_t all = (int64_t)(row[2 * (nbins - 1)] + row[2 * (nbins - 1) + 1]);
            side = all - left < left ? 1u : 0u;
        }
        s_side[k] = (uint8_t)side;
        if (blockIdx.x == 0 && pick) lside[k] = side;
    }
    if (wave == nwaves - 1) {
        // caps and starts of the lists: an exclusive scan of the caps
        uint32_t cap = 0u;
        if (lane < nslots) cap = cap_prev ? cap_prev[sib ? lane : lane >> 1] : cap_root;
        uint32_t x = cap;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const uint32_t y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (lane < nslots) {
            s_start[lane] = x - cap;
            s_cap[lane] = cap;
            if (blockIdx.x == 0) {
                lstart[lane] = x - cap;
                lcap[lane] = cap;
            }
        }
        s_cnt[lane] = 0u;
    }
    __syncthreads();

    // per event of the thread's steps: node << 16 | rank within the
    // workgroup's entries of that node, or ~0 (no entry)
    constexpr int STEPS = route_list_steps<SIGNED, OFF32>();
    constexpr int64_t EVENTS = route_list_events<SIGNED, OFF32>();
    uint32_t rec[STEPS][kHistE];
    uint32_t negs[STEPS];
    // the workgroups on XCD x = blockIdx % 8 take the events [x R, (x + 1) R)
    // (the range every per-event pass of the fit gives that XCD), in turn
    const int64_t xlo = (int64_t)(blockIdx.x % kXcds) * xcd_events;
    const int64_t base_i = xlo + (int64_t)(blockIdx.x / kXcds) * EVENTS;
    const int64_t end_i = min(min(n, xlo + xcd_events), base_i + EVENTS);
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
        const int64_t i0 = base_i + ((int64_t)st * kRouteListThreads + threadIdx.x) * kHistE;
        negs[st] = 0u;
#pragma unroll
        for (int e = 0; e < kHistE; ++e) rec[st][e] = ~0u;
        if (i0 < end_i) {
            const uint2 pin = node_in ? *reinterpret_cast<const uint2 *>(node_in + i0)
                                      : make_uint2(0x01010101u, 0x01010101u);
            // the parents are taken from pin again below rather than held
            uint32_t code[kHistE];
#pragma unroll
            for (int e = 0; e < kHistE; ++e) {
                const uint32_t k = byte8(pin, e) - half;
                const uint32_t kk = k < half ? k : 0u;
                code[e] = OFF32 ? xb[(uint32_t)min((int)s_cf[kk], d - 1) * (uint32_t)ldb +
                                     (uint32_t)(i0 + e)]
                                : xb[(int64_t)min((int)s_cf[kk], d - 1) * ldb + i0 + e];
            }
            const uint4 wx = reinterpret_cast<const uint4 *>(w + i0)[0];
            const uint4 wy = reinterpret_cast<const uint4 *>(w + i0)[1];
            const uint32_t wb[kHistE] = {wx.x, wx.y, wx.z, wx.w, wy.x, wy.y, wy.z, wy.w};
            uint2 vs = make_uint2(0u, 0u);
            if (SIGNED) vs = *reinterpret_cast<const uint2 *>(vsign + i0);
            uint32_t o[2] = {0u, 0u};
            uint32_t below = 0u;
#pragma unroll
            for (int e = 0; e < kHistE; ++e) {
                uint32_t p = byte8(pin, e), kk = p - half;
                bool stop = false, earlier = false;
                if (kk >= half) {
                    earlier = miss & (p < half);
                    stop = earlier;
                    if (!earlier) eflag |= kErrRoute;
                    kk = 0u;
                    p = earlier ? p : half;
                }
                stop |= miss & (code[e] == (uint32_t)kMissingCode);
                const uint32_t ne = stop ? p : 2u * p + (code[e] >= s_cc[kk] ? 1u : 0u);
                o[e >> 2] |= ne << (8 * (e & 3));
                const uint32_t ab = wb[e] & 0x7fffffffu;
                if (ab != 0u && !stop) {
                    // an entry of its list if its node is listed and its
                    // weight on the grid
                    const uint32_t nl = ne - nodes;
                    const bool listed = !pick || (nl & 1u) == s_side[kk];
                    if (ab < tau_bits) below |= 1u << e;
                    if (listed && ab >= tau_bits) {
                        const uint32_t slot = sib ? kk : stops ? 2u * kk : nl;
                        rec[st][e] = slot << 16 | atomicAdd(&s_cnt[slot], 1u);
                    }
                } else if (stops && stop && !earlier && ab >= tau_bits) {
                    // stops at parent kk here: its list of stopped events
                    rec[st][e] = (2u * kk + 1u) << 16 | atomicAdd(&s_cnt[2u * kk + 1u], 1u);
                }
                if (SIGNED && byte8(vs, e)) negs[st] |= 1u << e;
            }
            *reinterpret_cast<uint2 *>(node_out + i0) = make_uint2(o[0], o[1]);
            if (below) {   // rare: weights below the grid, every feature's side histogram
                for (int e = 0; e < kHistE; ++e) {
                    if (!((below >> e) & 1u)) continue;
                    const uint32_t ne = byte8(make_uint2(o[0], o[1]), e);
                    const uint32_t bits = __float_as_uint(w[i0 + e]);
                    double wa = (double)__uint_as_float(bits & 0x7fffffffu);
                    if ((negs[st] >> e) & 1u) wa = -wa;
                    for (int j = 0; j < d; ++j) {
                        const uint32_t bin = xb[(int64_t)j * ldb + i0 + e];
                        if (bin < (uint32_t)nbins) {
                            const size_t gi =
                                ((((size_t)(ne - nodes) * d + j) * nbins + bin) * 2) + (bits >> 31);
                            atomicAdd(&small[gi], wa);
                        } else if (!(miss && bin == (uint32_t)kMissingCode)) {
                            eflag |= kErrBin;
                        }
                    }
                }
                atomicOr(sany, 1u);
            }
        }
    }
    __syncthreads();
    // workgroup 0 records the parents' cuts in the model (the gain's load in
    // flight with the reservation)
    const bool crec = pwave && blockIdx.x == 0 && rec_f;
    const double rg = crec ? record_parent_cut(s_cf, s_cc, lane, d, cslices, cand_gain, rec_f,
                                               rec_c) : 0.0;
    if (threadIdx.x < (unsigned)nslots) {
        const uint32_t c = s_cnt[threadIdx.x];
        s_base[threadIdx.x] = c ? atomicAdd(&cursor[threadIdx.x], c) : 0u;
    }
    __syncthreads();
#pragma unroll
    for (int st = 0; st < STEPS; ++st) {
        const int64_t i0 = base_i + ((int64_t)st * kRouteListThreads + threadIdx.x) * kHistE;
        if (i0 < end_i) {
            // the weights again (in L2), rather than held in registers across
            // the reservation
            const uint4 wx = reinterpret_cast<const uint4 *>(w + i0)[0];
            const uint4 wy = reinterpret_cast<const uint4 *>(w + i0)[1];
            const uint32_t wb[kHistE] = {wx.x, wx.y, wx.z, wx.w, wy.x, wy.y, wy.z, wy.w};
#pragma unroll
            for (int e = 0; e < kHistE; ++e) {
                const uint32_t r = rec[st][e];
                if (r != ~0u) {
                    const uint32_t slot = r >> 16;
                    const uint32_t pos = s_base[slot] + (r & 0xffffu);
                    // the caps bound every count; an entry beyond one is an error
                    if (pos < s_cap[slot])
                        list[(size_t)s_start[slot] + pos] = make_uint2(
                            (uint32_t)(i0 + e) | (((negs[st] >> e) & 1u) << 31), wb[e]);
                    else
                        eflag |= kErrRoute;
                }
            }
        }
    }
    if (crec) rec_g[lane] = rg;
    if (eflag) atomicOr(err, eflag);
}

// Histogram pass over the lists of route_list_kernel: with lmode
// kCutSibling one child of every parent (lside[k] = 1: the right one; the
// cut scan forms the other as parent - child), with kCutStopped that child
// and the events that stopped at the parent (lists 2k and 2k + 1), with
// kCutPlain every node of the layer.  Each feature group's `parts` workgroups (parts > lists) share
// the entries of those lists: with E entries in all, list k of m_k entries
// gets C_k = ceil(m_k / ceil(E / (parts - lists))) equal parts (none when
// empty), numbered from base_k = C_0 + ... + C_(k-1); the C_k add up to at
// most parts.  Workgroup 0 records {base_k, C_k | flag << 31} in lchunks
// for the cut scan.  Workgroup (part, feature group g) adds its part of its list
// for the features [g FPG, g FPG + FPG) into its LDS rows (one per feature,
// 256 bins x 2 classes of 64-bit fixed-point counters, as in the streaming
// pass); each entry's codes are FPG / 4 words of the event's row in xr
// (stride dr).  Every entry is on the grid (route_list_kernel sends the
// others to the side histogram).  Rows are written out prefix-summed to
// partial[base_k + part][feature][bin][class].  The feature groups of one
// part run on one XCD, so that the event rows the first reads are in that
// XCD's L2 for the others.
template <int FPG, bool SIGNED>
__global__ __launch_bounds__(1024) void hist_list_kernel(
    const uint2 *__restrict__ list, const uint32_t *__restrict__ lstart,
    const uint32_t *__restrict__ lcap, const uint32_t *__restrict__ cursor,
    const uint32_t *__restrict__ lside, const uint8_t *__restrict__ xr, int dr, int d,
    int nbins, bool miss, int G, int parts, int nlists, int lmode, int per_xcd, int scale,
    int copies, int copy_stride, uint2 *__restrict__ lchunks, uint64_t *__restrict__ partial,
    int *__restrict__ err, uint32_t *__restrict__ cnt_out) {
    constexpr int NQ = FPG / 4;
    // the rows take all of the LDS (40 features: 160 KiB); the prologue's
    // few words sit at its start until the rows are cleared
    extern __shared__ uint64_t lds[];
    uint32_t *hdr = reinterpret_cast<uint32_t *>(lds);
    const int q = (blockIdx.x % kXcds) * per_xcd + blockIdx.x / kXcds;
    const int lane = threadIdx.x % kWave, wave = threadIdx.x / kWave;
    const int w = q / G;   // part slot of this workgroup
    if (wave == 0) {
        // list k's length, first entry and flag; parts per list from the total
        uint32_t m = 0u, first = 0u, flag = 0u;
        if (lane < nlists) {
            m = min(cursor[lane], lcap[lane]);
            first = lstart[lane];
            flag = lmode == kCutSibling                         ? lside[lane]
                   : lmode == kCutStopped && (lane & 1) == 0 ? lside[lane >> 1]
                                                             : 0u;
        }
        uint64_t tot = m;
#pragma unroll
        for (int o = kWave / 2; o > 0; o >>= 1) tot += __shfl_xor(tot, o);
        const uint64_t target = tot > 0 ? (tot + (parts - nlists) - 1) / (parts - nlists) : 1;
        const uint32_t c = (uint32_t)((m + target - 1) / target);
        uint32_t x = c;
#pragma unroll
        for (int o = 1; o < kWave; o <<= 1) {
            const uint32_t y = __shfl_up(x, o);
            if (lane >= o) x += y;
        }
        if (lane < nlists && blockIdx.x == 0) lchunks[lane] = make_uint2(x - c, c | flag << 31);
        if (cnt_out && blockIdx.x == 0) {
            // bounds on the on-grid sampled events of every node of the layer
            // (the next layer's list capacities; entries never leave them):
            // a listed node's entries, and for the other child of a parent
            // the parent's capacity minus the listed child's entries (and
            // minus the events that stopped at the parent)
            const uint32_t m_next = __shfl_down(m, 1);
            if (lmode == kCutPlain) {
                if (lane < nlists) cnt_out[lane] = m;
            } else if (lmode == kCutSibling) {
                if (lane < nlists) {
                    const uint32_t cap = lcap[lane];
                    cnt_out[2 * lane + flag] = m;
                    cnt_out[2 * lane + 1 - flag] = cap - m;
                }
            } else if (lane < nlists && (lane & 1) == 0) {   // kCutStopped: lists 2k, 2k + 1
                const uint32_t cap = lcap[lane];
                const int k = lane >> 1;
                cnt_out[2 * k + flag] = m;
                cnt_out[2 * k + 1 - flag] = cap - m - m_next;
            }
        }
        // the list whose parts hold part slot w, if any
        const bool mine = lane < nlists && (uint32_t)w >= x - c && (uint32_t)w < x;
        const uint64_t any = __ballot(mine);   // every lane of the wavefront votes
        if (lane == 0) hdr[0] = any != 0ull ? 1u : 0u;
        if (mine) {
            hdr[1] = w - (x - c);   // part within the list
            hdr[2] = c;
            hdr[3] = m;
            hdr[4] = first;
            hdr[5] = x - c;
        }
    }
    __syncthreads();
    const bool used = hdr[0] != 0u && q < G * parts;
    const uint32_t c = hdr[1], pbase = hdr[5];
    const uint64_t m = hdr[3], C = hdr[2], first = hdr[4];
    __syncthreads();   // the header is read before the rows are cleared over it
    if (!used) return;   // an unused part slot
    const int g = q % G;
    const int j0 = g * FPG;
    const int nf = min(FPG, d - j0);
    const int qbase = j0 / 4, qmax = dr / 4 - 1;
    const int lds_n = FPG * kRow;
    uint64_t *const lds_lane = reinterpret_cast<uint64_t *>(
        reinterpret_cast<char *>(lds) + (lane & (copies - 1)) * copy_stride);
    {
        uint4 *l4 = reinterpret_cast<uint4 *>(lds);
        const int n16 = copies > 1 ? copies * copy_stride / 16 : lds_n / 2;
        for (int t = threadIdx.x; t < n16; t += blockDim.x) l4[t] = make_uint4(0u, 0u, 0u, 0u);
    }
    const int64_t lo = (int64_t)(first + m * c / C);
    const int64_t hi = (int64_t)(first + m * (c + 1) / C);
    const int64_t T = blockDim.x;
    lds_barrier();

    char *ldsb = reinterpret_cast<char *>(lds_lane);
    auto add = [&](const uint2 en, const uint32_t (&cw)[NQ]) {
        const uint32_t bits = en.y;
        const uint32_t ab = bits & 0x7fffffffu;
        const int sh = (int)(ab >> 23) - 150 + scale;   // >= 0 on the grid
        uint64_t fx = (uint64_t)((ab & 0x7fffffu) | 0x800000u) << sh;
        if (SIGNED && (en.x >> 31)) fx = 0ull - fx;
        const uint32_t base = (bits >> 28) & 8u;
#pragma unroll
        for (int ff = 0; ff < FPG; ++ff) {
            if (ff < nf) {   // (uniform) the last group may hold fewer features
                const uint32_t off = base + (((cw[ff >> 2] >> (8 * (ff & 3))) & 0xffu) << 4);
                atomicAdd(reinterpret_cast<uint64_t *>(ldsb + off) + ff * kRow, fx);
            }
        }
    };
    // a group that starts the row and whose words fit it reads them as
    // 16-byte words (rows are a multiple of 16 bytes long)
    constexpr int NV = (NQ + 3) / 4;
    const bool vec = j0 == 0 && NV * 16 <= dr;
    auto codes = [&](const uint2 en, uint32_t (&cw)[NQ]) {
        const uint8_t *rb = xr + (size_t)(en.x & 0x7fffffffu) * dr;
        if (vec) {
            uint4 v[NV];
#pragma unroll
            for (int i = 0; i < NV; ++i) v[i] = reinterpret_cast<const uint4 *>(rb)[i];
#pragma unroll
            for (int qq = 0; qq < NQ; ++qq) {
                const uint4 &u = v[qq >> 2];
                cw[qq] = (qq & 3) == 0 ? u.x : (qq & 3) == 1 ? u.y : (qq & 3) == 2 ? u.z : u.w;
            }
        } else {
            const uint32_t *row = reinterpret_cast<const uint32_t *>(rb);
#pragma unroll
            for (int qq = 0; qq < NQ; ++qq) cw[qq] = row[min(qbase + qq, qmax)];
        }
    };
    // two entries per thread and step; the next step's entries are loaded
    // while this step's codes arrive and are added
    int64_t ja = lo + threadIdx.x;
    uint2 ea = make_uint2(0u, 0u), eb = make_uint2(0u, 0u);
    if (ja < hi) ea = list[ja];
    if (ja + T < hi) eb = list[ja + T];
    while (ja < hi) {
        const bool has_b = ja + T < hi;
        uint32_t ca[NQ], cb[NQ];
        codes(ea, ca);
        if (has_b) codes(eb, cb);
        const int64_t jn = ja + 2 * T;
        uint2 na = make_uint2(0u, 0u), nb = make_uint2(0u, 0u);
        if (jn < hi) na = list[jn];
        if (jn + T < hi) nb = list[jn + T];
        add(ea, ca);
        if (has_b) add(eb, cb);
        ja = jn;
        ea = na;
        eb = nb;
    }
    lds_barrier();
    int eflag = 0;
    hist_write_rows(lds, copies, copy_stride, lds_n, 1, nf, FPG, 0, j0, 1, d, nbins, miss, true,
                    reinterpret_cast<uint4 *>(partial + (size_t)(pbase + c) * d * nbins * 2),
                    eflag);
    if (eflag) atomicOr(err, eflag);
}

// node <- 2 node + [xb[f][i] >= c] with (f, c) the cut of the node.
__global__ __launch_bounds__(256) void route_kernel(const uint8_t *__restrict__ xb, int64_t ldb,
                                                    int64_t n, int d, uint8_t *__restrict__ node,
                                                    const uint8_t *__restrict__ cut_f,
                                                    const uint8_t *__restrict__ cut_c, int layer,
                                                    int *__restrict__ err) {
    const int lo = 1 << layer;
    int eflag = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int nd = node[i];
        const unsigned k = (unsigned)(nd - lo);
        if (k >= (unsigned)lo) {
            eflag |= kErrRoute;
            continue;
        }
        const int f = cut_f[k];
        if (f >= d) {
            eflag |= kErrRoute;
            continue;
        }
        node[i] = (uint8_t)(2 * nd + (xb[(int64_t)f * ldb + i] >= cut_c[k] ? 1 : 0));
    }
    if (eflag) atomicOr(err, eflag);
}

// ---------------------------------------------------------------------------
// Forest traversal.  A workgroup stages a tile of `blockDim.x` events (all
// model features, padded rows to spread LDS banks) and a chunk of trees in
// LDS; each thread walks its event through every tree (left = bin < cut,
// Fig. 1), adds the leaf's boost weight to F in float64 in tree order, and
// writes 1 / (1 + exp(-2F)) as float32.
__global__ __launch_bounds__(1024) void apply_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d_used,
    const uint16_t *__restrict__ cuts, const double *__restrict__ leaves, int T, int depth,
    bool missing, int tpc, double f0, float *__restrict__ prob, double *__restrict__ score) {
    extern __shared__ double smem[];
    const int nin = (1 << depth) - 1;
    // boost weights per tree: the leaves, or with missing values (section
    // 4.2) every node in heap order, for events that stop at an inner node
    const int nleaf = missing ? 2 * nin + 1 : 1 << depth;
    const int first_id = missing ? 1 : 1 << depth;
    double *s_leaf = smem;
    uint16_t *s_cut = reinterpret_cast<uint16_t *>(s_leaf + (size_t)tpc * nleaf);
    uint8_t *s_x = reinterpret_cast<uint8_t *>(s_cut + (((size_t)tpc * nin + 3) & ~(size_t)3));
    const int XS = blockDim.x + 4;
    const int nchunks = (T + tpc - 1) / tpc;
    const int64_t ntiles = (n + blockDim.x - 1) / blockDim.x;
    bool staged = false;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t i = tile * blockDim.x + threadIdx.x;
        __syncthreads();
        for (int f = 0; f < d_used; ++f)
            s_x[f * XS + threadIdx.x] = i < n ? xb[(int64_t)f * ldb + i] : 0;
        double Fv = f0;
        for (int ch = 0; ch < nchunks; ++ch) {
            const int t0 = ch * tpc;
            const int tc = min(tpc, T - t0);
            if (nchunks > 1 || !staged) {
                __syncthreads();
                for (int q = threadIdx.x; q < tc * nleaf; q += blockDim.x)
                    s_leaf[q] = leaves[(size_t)t0 * nleaf + q];
                for (int q = threadIdx.x; q < tc * nin; q += blockDim.x)
                    s_cut[q] = cuts[(size_t)t0 * nin + q];
                staged = true;
            }
            __syncthreads();
            for (int t = 0; t < tc; ++t) {
                int node = 1;
                for (int lvl = 0; lvl < depth; ++lvl) {
                    const uint16_t cc = s_cut[t * nin + node - 1];
                    const int f = cc & 0xff;
                    const int c = cc >> 8;
                    const int code = s_x[f * XS + threadIdx.x];
                    if (missing && code == kMissingCode) break;   // stops at this node
                    node = 2 * node + (code >= c ? 1 : 0);
                }
                Fv += s_leaf[t * nleaf + node - first_id];
            }
        }
        if (i < n) {
            prob[i] = (float)(1.0 / (1.0 + exp(-2.0 * Fv)));
            if (score) score[i] = Fv;
        }
    }
}

// ---------------------------------------------------------------------------
// Bin code of a float: number of boundaries <= value (upper bound by binary
// search over the feature's boundaries in LDS).  Row padding [n, ldb) is
// written as 0.
// Forest traversal for depth <= 3 (the apply workload's forests).  Every
// thread scores two adjacent events.  The 2^D - 1 cuts of a tree are uniform
// across the workgroup, so they come as scalar loads of a per-tree record of
// 16 words: for heap node k + 1, word k = the LDS offset of its feature's row
// in the code tile (feature * XS) and word 8 + k = (256 - bin) * 0x10001.  All
// cuts' codes of both events are read up front (one 16-bit LDS read per cut,
// no chain from one level to the next); v_perm puts the two codes in the low
// bytes of the two 16-bit halves, and adding word 8 + k sets bit 8 (first
// event) and bit 24 (second event) exactly when code >= bin (right child).
// The path is then bitfield selects on those words for both events at once,
// and each reached leaf's value is one LDS read, added to F in tree order.
// Leaf values of tpc trees at a time are staged in LDS (all of them when they
// fit), the codes of a tile of 2 * blockDim events per feature (row stride XS
// = 2 * blockDim + 8).
constexpr int kApplyBatch = 4;

// Leaf indices of the two events in a tree of depth D <= 3: the first in
// bits 0..2, the second in bits 16..18.
template <int D>
__device__ __forceinline__ uint32_t shallow_leaf2(const uint8_t *xpair, const uint32_t *off,
                                                  const uint32_t *add) {
    constexpr int NIN = (1 << D) - 1;
    uint32_t w[NIN];
#pragma unroll
    for (int k = 0; k < NIN; ++k) {
        const uint32_t p = *reinterpret_cast<const uint16_t *>(xpair + off[k]);
        w[k] = __builtin_amdgcn_perm(p, p, 0x0c010c00u) + add[k];
    }
    constexpr uint32_t kBits = 0x01000100u;   // the decision bits (8 and 24)
    const uint32_t r1 = w[0];
    if (D == 1) return (r1 & kBits) >> 8;
    const uint32_t r2 = (r1 & w[2]) | (~r1 & w[1]);   // child of the root reached
    if (D == 2) return ((r1 & kBits) >> 7) | ((r2 & kBits) >> 8);
    const uint32_t t0 = (r2 & w[4]) | (~r2 & w[3]);
    const uint32_t t1 = (r2 & w[6]) | (~r2 & w[5]);
    const uint32_t r3 = (r1 & t1) | (~r1 & t0);
    return ((r1 & kBits) >> 6) | ((r2 & kBits) >> 7) | ((r3 & kBits) >> 8);
}

// With FLOATS the tile is staged from float32 values (section 2.2's
// inverse transform, fused): ftab holds, per feature, the ascending distinct
// thresholds that the forest's cuts on it test (offsets [d_used + 1], then
// the thresholds' float bits), and a value's code is the number of those
// thresholds at or below it, found by a binary search in LDS; the node
// records then carry, instead of the bin c, the rank c' of the node's
// threshold among its feature's (code >= c' exactly when x >= threshold).
// NaN compares false with every threshold: code 0, the left branch of every
// cut, as the threshold test gives.
template <int D, bool FLOATS>
__global__ __launch_bounds__(1024) void apply_shallow_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, const float *__restrict__ xf, int64_t ldx,
    const uint32_t *__restrict__ ftab, int ftab_words, int64_t n, int d_used,
    const uint32_t *__restrict__ nodes, const double *__restrict__ leaves, int T, int tpc,
    double f0, float *__restrict__ prob, double *__restrict__ score) {
    constexpr int NLEAF = 1 << D;
    constexpr int NIN = (1 << D) - 1;
    extern __shared__ double smem[];
    double *s_leaf = smem;   // [tpc][NLEAF]
    uint8_t *s_x = reinterpret_cast<uint8_t *>(s_leaf + (size_t)tpc * NLEAF);   // [d_used][XS]
    const int tile_events = 2 * blockDim.x;
    const int XS = tile_events + 8;   // the stride the node records were prepared for
    // FLOATS: thresholds per feature, after the code tile (XS is a multiple of 8)
    uint32_t *s_tab = reinterpret_cast<uint32_t *>(s_x + (size_t)d_used * XS);
    const float *s_thr = reinterpret_cast<const float *>(s_tab + d_used + 1);
    if (FLOATS) {
        for (int q = threadIdx.x; q < ftab_words; q += blockDim.x) s_tab[q] = ftab[q];
    }
    const int nchunks = (T + tpc - 1) / tpc;
    const int64_t ntiles = (n + tile_events - 1) / tile_events;
    const uint8_t *xpair = s_x + 2 * threadIdx.x;
    bool staged = false;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t i0 = tile * tile_events + 2 * threadIdx.x;   // this thread's events
        __syncthreads();
        if (FLOATS) {
            // 8 features' values loaded at a time, then their codes searched
            for (int fb = 0; fb < d_used; fb += 8) {
                float va[8], vb[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const float *src = xf + (int64_t)min(fb + u, d_used - 1) * ldx + i0;
                    va[u] = i0 < n ? src[0] : 0.0f;
                    vb[u] = i0 + 1 < n ? src[1] : 0.0f;
                }
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    const int f = fb + u;
                    if (f >= d_used) break;
                    const int lo = (int)s_tab[f], m = (int)s_tab[f + 1] - lo;
                    int ca = 0, cb = 0;
                    // count of thresholds <= value (binary lifting over m entries)
                    for (int step = m > 0 ? 1 << (31 - __clz(m)) : 0; step > 0; step >>= 1) {
                        const int ta = ca + step, tb = cb + step;
                        if (ta <= m && s_thr[lo + ta - 1] <= va[u]) ca = ta;
                        if (tb <= m && s_thr[lo + tb - 1] <= vb[u]) cb = tb;
                    }
                    *reinterpret_cast<uint16_t *>(s_x + f * XS + 2 * threadIdx.x) =
                        (uint16_t)(ca | (cb << 8));
                }
            }
        } else {
            for (int f = 0; f < d_used; ++f) {
                const uint8_t *src = xb + (int64_t)f * ldb + i0;
                uint16_t pair = 0;
                if (i0 + 1 < n)
                    pair = *reinterpret_cast<const uint16_t *>(src);
                else if (i0 < n)
                    pair = src[0];
                *reinterpret_cast<uint16_t *>(s_x + f * XS + 2 * threadIdx.x) = pair;
            }
        }
        double Fa = f0, Fb = f0;
        for (int ch = 0; ch < nchunks; ++ch) {
            const int t0 = ch * tpc;
            const int tc = min(tpc, T - t0);
            if (nchunks > 1 || !staged) {
                __syncthreads();
                for (int q = threadIdx.x; q < tc * NLEAF; q += blockDim.x)
                    s_leaf[q] = leaves[(size_t)t0 * NLEAF + q];
                staged = true;
            }
            __syncthreads();
            // full batches of kApplyBatch trees: every load of the batch (node
            // records, codes, leaf values) is issued before its results are
            // used, then the leaf values are added in tree order
            int t = 0;
            for (; t + kApplyBatch <= tc; t += kApplyBatch) {
                uint32_t off[kApplyBatch][NIN], add[kApplyBatch][NIN];
#pragma unroll
                for (int u = 0; u < kApplyBatch; ++u) {
                    const uint32_t *nt = nodes + (size_t)(t0 + t + u) * 16;
#pragma unroll
                    for (int k = 0; k < NIN; ++k) {
                        off[u][k] = nt[k];
                        add[u][k] = nt[8 + k];
                    }
                }
                uint32_t idx[kApplyBatch];
#pragma unroll
                for (int u = 0; u < kApplyBatch; ++u) idx[u] = shallow_leaf2<D>(xpair, off[u], add[u]);
                double la[kApplyBatch], lb[kApplyBatch];
#pragma unroll
                for (int u = 0; u < kApplyBatch; ++u) {
                    const double *lt = s_leaf + (t + u) * NLEAF;
                    la[u] = lt[idx[u] & 0xffffu];
                    lb[u] = lt[idx[u] >> 16];
                }
#pragma unroll
                for (int u = 0; u < kApplyBatch; ++u) {
                    Fa += la[u];
                    Fb += lb[u];
                }
            }
            for (; t < tc; ++t) {
                const uint32_t *nt = nodes + (size_t)(t0 + t) * 16;
                uint32_t off[NIN], add[NIN];
#pragma unroll
                for (int k = 0; k < NIN; ++k) {
                    off[k] = nt[k];
                    add[k] = nt[8 + k];
                }
                const uint32_t idx = shallow_leaf2<D>(xpair, off, add);
                const double *lt = s_leaf + t * NLEAF;
                Fa += lt[idx & 0xffffu];
                Fb += lt[idx >> 16];
            }
        }
        if (i0 < n) {
            prob[i0] = (float)(1.0 / (1.0 + exp(-2.0 * Fa)));
            if (score) score[i0] = Fa;
        }
        if (i0 + 1 < n) {
            prob[i0 + 1] = (float)(1.0 / (1.0 + exp(-2.0 * Fb)));
            if (score) score[i0 + 1] = Fb;
        }
    }
}

// Importance of every feature for every event (section 4.3): each node on
// an event's path adds its separation gain to the importance of the node's
// cut feature, tree by tree in float64.  A workgroup stages a tile of codes
// (one event per thread) and chunks of the forest (packed cut and gain) in
// LDS; each thread keeps its event's accumulators in an LDS column.
__global__ __launch_bounds__(256) void importance_kernel(
    const uint8_t *__restrict__ xb, int64_t ldb, int64_t n, int d_used,
    const uint16_t *__restrict__ cuts, const double *__restrict__ gains, int T, int depth,
    bool missing, int tpc, double *__restrict__ imp, int64_t ldi, int d_out) {
    extern __shared__ double smem[];
    const int nin = (1 << depth) - 1;
    const int nt = blockDim.x;
    double *s_gain = smem;                            // [tpc][nin]
    double *s_acc = s_gain + (size_t)tpc * nin;       // [d_used][nt]
    uint16_t *s_cut = reinterpret_cast<uint16_t *>(s_acc + (size_t)d_used * nt);   // [tpc][nin]
    uint8_t *s_x = reinterpret_cast<uint8_t *>(s_cut + (((size_t)tpc * nin + 3) & ~(size_t)3));
    const int XS = nt + 4;
    const int nchunks = (T + tpc - 1) / tpc;
    const int64_t ntiles = (n + nt - 1) / nt;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t i = tile * nt + threadIdx.x;
        __syncthreads();
        for (int f = 0; f < d_used; ++f) {
            s_x[f * XS + threadIdx.x] = i < n ? xb[(int64_t)f * ldb + i] : 0;
            s_acc[f * nt + threadIdx.x] = 0.0;
        }
        for (int ch = 0; ch < nchunks; ++ch) {
            const int t0 = ch * tpc;
            const int tc = min(tpc, T - t0);
            __syncthreads();
            for (int q = threadIdx.x; q < tc * nin; q += nt) {
                s_gain[q] = gains[(size_t)t0 * nin + q];
                s_cut[q] = cuts[(size_t)t0 * nin + q];
            }
            __syncthreads();
            for (int t = 0; t < tc; ++t) {
                int node = 1;
                for (int lvl = 0; lvl < depth; ++lvl) {
                    const int k = t * nin + node - 1;
                    const uint16_t cc = s_cut[k];
                    const int f = cc & 0xff;
                    const int code = s_x[f * XS + threadIdx.x];
                    if (missing && code == kMissingCode) break;   // the cut does not apply
                    s_acc[f * nt + threadIdx.x] += s_gain[k];
                    node = 2 * node + (code >= (cc >> 8) ? 1 : 0);
                }
            }
        }
        if (i < n)
            for (int f = 0; f < d_out; ++f)
                imp[(int64_t)f * ldi + i] = f < d_used ? s_acc[f * nt + threadIdx.x] : 0.0;
    }
}

// Forest traversal of float32 events with value thresholds (section 2.2:
// the cut "bin >= c" of feature j is the test x >= b_j,c, the c-th training
// boundary, since a value's bin counts the boundaries at or below it), for
// trees deeper than kApplyShallowDepth or with missing values.  A workgroup
// stages a tile of one event per thread, feature-major, in LDS, and chunks
// of the forest's records rec: [T][2^D - 1] pairs (feature, threshold bits);
// each event walks its path.
template <int D>
__global__ __launch_bounds__(1024) void apply_float_kernel(
    const float *__restrict__ x, int64_t ldx, int64_t n, int d_used,
    const uint2 *__restrict__ rec, const double *__restrict__ leaves, int T, bool missing,
    int tpc, double f0, float *__restrict__ prob, double *__restrict__ score) {
    constexpr int NIN = (1 << D) - 1;
    // boost weights per tree: the leaves, or with missing values every node
    // in heap order (a NaN value stops its event at the node cutting on it)
    const int NLEAF = missing ? 2 * NIN + 1 : 1 << D;
    const int first_id = missing ? 1 : 1 << D;
    extern __shared__ double smem[];
    double *s_leaf = smem;                                                    // [tpc][NLEAF]
    uint2 *s_rec = reinterpret_cast<uint2 *>(s_leaf + (size_t)tpc * NLEAF);   // [tpc][NIN]
    float *s_x = reinterpret_cast<float *>(s_rec + (size_t)tpc * NIN);
    const int XS = blockDim.x;   // [d_used][XS]
    const int nchunks = (T + tpc - 1) / tpc;
    const int64_t ntiles = (n + blockDim.x - 1) / blockDim.x;
    const float *xme = s_x + threadIdx.x;
    bool staged = false;
    for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
        const int64_t i = tile * blockDim.x + threadIdx.x;
        __syncthreads();
        for (int f = 0; f < d_used; ++f) s_x[f * XS + threadIdx.x] = i < n ? x[(int64_t)f * ldx + i] : 0.0f;
        double Fv = f0;
        for (int ch = 0; ch < nchunks; ++ch) {
            const int t0 = ch * tpc;
            const int tc = min(tpc, T - t0);
            if (nchunks > 1 || !staged) {
                __syncthreads();
                for (int q = threadIdx.x; q < tc * NLEAF; q += blockDim.x)
                    s_leaf[q] = leaves[(size_t)t0 * NLEAF + q];
                for (int q = threadIdx.x; q < tc * NIN; q += blockDim.x) {
                    const uint2 r = rec[(size_t)t0 * NIN + q];
                    s_rec[q] = make_uint2(r.x * (uint32_t)XS, r.y);   // row offset
                }
                staged = true;
            }
            __syncthreads();
            for (int t = 0; t < tc; ++t) {
                int node = 1;
#pragma unroll
                for (int lvl = 0; lvl < D; ++lvl) {
                    const uint2 r = s_rec[t * NIN + node - 1];
                    const float xv = xme[r.x];
                    if (missing && xv != xv) break;   // NaN: stops at this node
                    node = 2 * node + (xv >= __uint_as_float(r.y) ? 1 : 0);
                }
                Fv += s_leaf[t * NLEAF + node - first_id];
            }
        }
        if (i < n) {
            prob[i] = (float)(1.0 / (1.0 + exp(-2.0 * Fv)));
            if (score) score[i] = Fv;
        }
    }
}

__global__ __launch_bounds__(256) void encode_kernel(const float *__restrict__ x, int64_t ldx,
                                                     int64_t n, int d,
                                                     const float *__restrict__ bounds, int nbins,
                                                     uint8_t *__restrict__ xb, int64_t ldb,
                                                     int *__restrict__ err) {
    __shared__ float sb[256];
    const int j = blockIdx.y;
    const int nb = nbins - 1;
    for (int k = threadIdx.x; k < nb; k += blockDim.x) sb[k] = bounds[(size_t)j * nb + k];
    __syncthreads();
    int eflag = 0;
    // the n codes of row j only: bytes of the row beyond n are not written
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        uint8_t code = 0;
        const float val = x[(int64_t)j * ldx + i];
        if (val != val) {
            // a missing value: the reserved code with at most 255 bins
            // (section 4.2), else an error
            if (nbins <= kMissingCode)
                code = (uint8_t)kMissingCode;
            else
                eflag |= kErrNan;
        } else {
            int lo = 0, len = nb;
            while (len > 0) {
                const int hh = len >> 1;
                if (sb[lo + hh] <= val) {
                    lo += hh + 1;
                    len -= hh + 1;
                } else {
                    len = hh;
                }
            }
            code = (uint8_t)lo;
        }
        xb[(int64_t)j * ldb + i] = code;
    }
    if (eflag) atomicOr(err, eflag);
}

}  // namespace

int64_t xcd_range(int64_t n) {
    const int64_t r = (n + kXcds - 1) / kXcds;
    return (r + kXcdQuantum - 1) / kXcdQuantum * kXcdQuantum;
}

namespace {

// Workgroups of a per-event pass: the same number on each XCD (a multiple
// of kXcds), at most one round of cu_count, as many as the XCD range needs.
int xcd_grid(int64_t n, int64_t events_per_block, int cu_count) {
    int64_t per = (xcd_range(n) + events_per_block - 1) / events_per_block;
    const int64_t cap = cu_count / kXcds > 0 ? cu_count / kXcds : 1;
    if (per > cap) per = cap;
    if (per < 1) per = 1;
    return (int)(kXcds * per);
}

int grid_for(int64_t n, int threads, int cap) {
    int64_t g = (n + threads - 1) / threads;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

// Raises a kernel's dynamic-LDS limit to what the device allows beside the
// kernel's static LDS.
template <typename K>
hipError_t allow_lds(K kernel, size_t max_lds) {
    if (max_lds <= kHistStaticLdsReserve) return hipSuccess;
    return hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                               hipFuncAttributeMaxDynamicSharedMemorySize,
                               (int)(max_lds - kHistStaticLdsReserve));
}

}  // namespace

// ===========================================================================
template <int FPG>
hipError_t allow_hist_lds(size_t max_lds) {
    const hipError_t e[] = {allow_lds(hist_kernel<false, 0, FPG, false, false>, max_lds),
                            allow_lds(hist_kernel<false, 0, FPG, true, false>, max_lds),
                            allow_lds(hist_kernel<true, 0, FPG, false, false>, max_lds),
                            allow_lds(hist_kernel<true, 1, FPG, false, false>, max_lds),
                            allow_lds(hist_kernel<true, 2, FPG, false, false>, max_lds),
                            allow_lds(hist_kernel<true, 4, FPG, false, false>, max_lds),
                            allow_lds(hist_kernel<true, 0, FPG, true, false>, max_lds),
                            allow_lds(hist_kernel<true, 1, FPG, true, false>, max_lds),
                            allow_lds(hist_kernel<true, 2, FPG, true, false>, max_lds),
                            allow_lds(hist_kernel<true, 4, FPG, true, false>, max_lds),
                            allow_lds(hist_kernel<true, 0, FPG, false, true>, max_lds),
                            allow_lds(hist_kernel<true, 1, FPG, false, true>, max_lds),
                            allow_lds(hist_kernel<true, 2, FPG, false, true>, max_lds),
                            allow_lds(hist_kernel<true, 4, FPG, false, true>, max_lds),
                            allow_lds(hist_kernel<true, 0, FPG, true, true>, max_lds),
                            allow_lds(hist_kernel<true, 1, FPG, true, true>, max_lds),
                            allow_lds(hist_kernel<true, 2, FPG, true, true>, max_lds),
                            allow_lds(hist_kernel<true, 4, FPG, true, true>, max_lds)};
    for (hipError_t x : e)
        if (x != hipSuccess) return x;
    return hipSuccess;
}

template <int FPG>
hipError_t allow_list_lds(size_t max_lds) {
    const hipError_t a = allow_lds(hist_list_kernel<FPG, false>, max_lds);
    return a != hipSuccess ? a : allow_lds(hist_list_kernel<FPG, true>, max_lds);
}

hipError_t prepare_kernels(size_t max_lds) {
    const hipError_t e[] = {allow_hist_lds<1>(max_lds), allow_hist_lds<2>(max_lds),
                            allow_hist_lds<4>(max_lds), allow_hist_lds<5>(max_lds),
                            allow_hist_lds<8>(max_lds), allow_lds(apply_kernel, max_lds),
                            allow_lds(leaf_kernel<false, 0>, max_lds),
                            allow_lds(leaf_kernel<true, 0>, max_lds),
                            allow_lds(leaf_kernel<true, 1>, max_lds),
                            allow_lds(leaf_kernel<true, 2>, max_lds),
                            allow_lds(leaf_kernel<true, 4>, max_lds),
                            allow_lds(apply_shallow_kernel<1, false>, max_lds),
                            allow_lds(apply_shallow_kernel<2, false>, max_lds),
                            allow_lds(apply_shallow_kernel<3, false>, max_lds),
                            allow_lds(apply_shallow_kernel<1, true>, max_lds),
                            allow_lds(apply_shallow_kernel<2, true>, max_lds),
                            allow_lds(apply_shallow_kernel<3, true>, max_lds),
                            allow_lds(apply_float_kernel<1>, max_lds),
                            allow_lds(apply_float_kernel<2>, max_lds),
                            allow_lds(apply_float_kernel<3>, max_lds),
                            allow_lds(apply_float_kernel<4>, max_lds),
                            allow_lds(apply_float_kernel<5>, max_lds),
                            allow_lds(apply_float_kernel<6>, max_lds),
                            allow_lds(apply_float_kernel<7>, max_lds),
                            allow_lds(importance_kernel, max_lds),
                            allow_lds(hist_reference_kernel, max_lds),
                            allow_list_lds<4>(max_lds), allow_list_lds<8>(max_lds),
                            allow_list_lds<12>(max_lds), allow_list_lds<20>(max_lds),
                            allow_list_lds<28>(max_lds), allow_list_lds<36>(max_lds),
                            allow_list_lds<40>(max_lds)};
    for (hipError_t x : e)
        if (x != hipSuccess) return x;
    return hipSuccess;
}

hipError_t launch_fill_u32(void *p, uint32_t value, size_t count, hipStream_t s) {
    if (count == 0) return hipSuccess;
    fill_u32_kernel<<<grid_for((int64_t)count, 256, 1024), 256, 0, s>>>(
        static_cast<uint32_t *>(p), value, count);
    return hipGetLastError();
}

hipError_t launch_validate(const int8_t *y, const float *v, int64_t n, double *class_partial,
                           int *err, hipStream_t s) {
    validate_kernel<<<kValidateBlocks, 256, 0, s>>>(y, v, n, class_partial, err);
    return hipGetLastError();
}

hipError_t launch_initial_score(const double *class_partial, double *f0, int *err,
                                hipStream_t s) {
    initial_score_kernel<<<1, 256, 0, s>>>(class_partial, kValidateBlocks, f0, err);
    return hipGetLastError();
}

hipError_t launch_tree_prep(const int8_t *y, const float *v, double *F, const double *f0,
                            const uint8_t *leaf_node, const double *leaf_prev,
                            const double *leaf_partial, int lblocks, double eta, double *leaf_rec,
                            int depth, bool missing, int64_t n, uint64_t seed, int tree,
                            double alpha, float *w, double *yts, double *score_out, int cu_count,
                            hipStream_t s) {
    if (leaf_partial && depth > kFusedLeafDepth) return hipErrorInvalidValue;
    tree_prep_kernel<<<xcd_grid(n, kLeafReduceThreads, cu_count), kLeafReduceThreads, 0, s>>>(
        y, v, F, f0, leaf_node, leaf_prev, leaf_partial, lblocks, eta, leaf_rec, depth, missing, n,
        seed, tree, alpha, w, yts, score_out, xcd_range(n));
    return hipGetLastError();
}

bool hist_fpg_supported(int f) {
    for (int c : kHistFpgSizes)
        if (c == f) return true;
    return false;
}

HistShape plan_histogram(int64_t n, int d, int n_bins, int layer, bool sibling, int cu_count,
                         size_t max_lds, const HistOverrides &ov) {
    const int fpg = ov.fpg, chunks = ov.chunks, threads = ov.threads;
    HistShape hs{};
    const int nodes = sibling && layer >= 1 ? 1 << (layer - 1) : 1 << layer;
    // an LDS row of one (node, feature) holds 256 bins x 2 classes
    const size_t per_node_feature = (size_t)kRowBytes;
    // the kernel's static LDS (cut table) shares the workgroup's LDS limit
    max_lds = max_lds > kHistStaticLdsReserve ? max_lds - kHistStaticLdsReserve : 0;
    int npg = (int)(max_lds / per_node_feature);
    if (npg < 1) npg = 1;
    if (npg > nodes) npg = nodes;
    hs.nodes_per_group = npg;
    hs.node_groups = (nodes + npg - 1) / npg;
    // Features per workgroup f (one of kHistFpgSizes) and event chunks per
    // XCD c8, from a cost model fitted to launches of this kernel on MI355X
    // (0.5M-10M events, 20-40 features, 1-16 histogrammed nodes).  The pass
    // is bound by LDS atomic issue: a ds_add_u64 wavefront instruction costs
    // ~9 clocks whether half or all of its lanes are active, so a workgroup
    // pays about kCostAdd us per thousand (event, feature) slots it streams,
    // sampled or not, counted or not, plus kCostEvent per thousand events;
    // the launch pays that once per round of workgroups, and every MB of
    // chunk partials written (and summed again by the cut scan) costs about
    // kCostPartial us.  With the CUs filled the slots per workgroup are about
    // equal for every f, so the model takes the fewest chunks (fewest
    // partials) that still fill the CUs, and it avoids node groups, which
    // stream every event once per group.
    const int t_threads = threads > 0 ? threads : 1024;
    const int64_t min_events = (int64_t)kHistE * t_threads;
    const int64_t R = xcd_range(n);
    const int64_t c8max = R / (min_events / 2) > 0 ? R / (min_events / 2) : 1;
    int f = 1;
    int64_t c8_pick = 0;
    if (fpg > 0) {
        f = fpg;
    } else {
        constexpr double kCostEvent = 0.01, kCostAdd = 0.057, kCostPartial = 0.25;
        double best = 0.0;
        for (int cand : kHistFpgSizes) {
            if (cand > d && cand != kHistFpgSizes[0]) continue;
            const int np = (int)std::min<size_t>((size_t)nodes, max_lds / ((size_t)cand * per_node_feature));
            if (np < 1) continue;
            const int ng = (nodes + np - 1) / np;
            const int g = ((d + cand - 1) / cand) * ng;
            int64_t top = cu_count / kXcds / g;
            if (top > c8max) top = c8max;
            if (top < 1) top = 1;
            for (int64_t c8 = 1; c8 <= top; ++c8) {
                const double ek = (double)((R + c8 - 1) / c8) / 1000.0;
                const int64_t wgs = kXcds * c8 * g;
                const double rounds = (double)((wgs + cu_count - 1) / cu_count);
                const double pmb = (double)(kXcds * c8) * nodes * d * n_bins * 16.0 / 1e6;
                const double t = rounds * ek * (kCostEvent + kCostAdd * cand) + kCostPartial * pmb;
                if (c8_pick == 0 || t < best) {
                    best = t;
                    f = cand;
                    c8_pick = c8;
                }
            }
        }
        if (chunks > 0) c8_pick = 0;
    }
    while (npg > 1 && (size_t)npg * f * per_node_feature > max_lds) --npg;
    hs.nodes_per_group = npg;
    hs.node_groups = (nodes + npg - 1) / npg;
    hs.features_per_group = f;
    hs.feature_groups = (d + f - 1) / f;
    hs.threads = t_threads;
    const int groups = hs.feature_groups * hs.node_groups;
    // Chunks: the same number in each XCD's event range [x R, (x + 1) R), so
    // that the workgroups of a chunk, which the launch places on that XCD,
    // read event data that the fit's other per-event passes wrote there (it
    // stays in the XCD's L2 across kernels).  At most one workgroup per CU
    // by default (a 1024-thread workgroup fills a CU): a few workgroups more
    // than CUs run as a second round and nearly double the pass; every extra
    // event chunk also adds one more partial histogram to write and to sum.
    int64_t c8 = chunks > 0 ? (chunks + kXcds - 1) / kXcds
               : c8_pick > 0 ? c8_pick : (int64_t)cu_count / kXcds / groups;
    if (chunks <= 0 && c8 > c8max) c8 = c8max;
    if (c8 > 255) c8 = 255;   // the kernel takes chunks per XCD in 8 bits
    if (c8 < 1) c8 = 1;
    int64_t ce = (R + c8 - 1) / c8;
    ce = (ce + kHistE - 1) / kHistE * kHistE;
    c8 = (R + ce - 1) / ce;
    hs.chunk_events = ce;
    hs.xcd_events = R;
    hs.chunks = (int)(kXcds * c8);
    hs.blocks = hs.chunks * groups;
    // LDS copies: up to 4 (as many as fit beside the node and feature choice
    // above) for long chunks, where they cut the serialization of lanes
    // that hit one counter (measured: -8% per pass on 10M events whose
    // discrete features hold <= 10 values, +4% on 0.5M-event passes, where
    // clearing and summing the copies is not amortised)
    const size_t one = (size_t)npg * f * per_node_feature;
    int copies = ov.copies > 0 ? ov.copies : (ce >= kHistCopiesMinEvents ? 4 : 1);
    while (copies > 1 && (size_t)copies * (one + kHistCopyShift) > max_lds) copies >>= 1;
    hs.copies = copies;
    hs.copy_stride = copies > 1 ? (int)(one + kHistCopyShift) : (int)one;
    hs.lds_bytes = copies > 1 ? (size_t)copies * hs.copy_stride : one;
    hs.sibling = sibling && layer >= 1;
    return hs;
}

int histogram_scale(double total_weight_bound) {
    if (!(total_weight_bound > 0.0) || !std::isfinite(total_weight_bound)) return 60;
    int e = 0;
    (void)std::frexp(total_weight_bound, &e);  // bound < 2^e
    int sc = 62 - e;                           // bound * 2^sc < 2^62
    if (sc > 60) sc = 60;
    if (sc < -60) sc = -60;
    return sc;
}

template <bool ROUTED, int NP, int FPG, bool SIGNED, bool MISS>
hipError_t launch_hist_np(const HistShape &hs, const uint8_t *xb, int64_t ldb, int64_t n, int d,
                          int n_bins, const uint8_t *node_in, uint8_t *node_out, const float *w,
                          const uint8_t *vsign, const ParentCuts &pc, int layer, int scale,
                          uint64_t *partial, double *small, int *err, unsigned long long *tl,
                          hipStream_t s) {
    const int cpx = hs.chunks / kXcds;
    if (d > 255 || hs.feature_groups > 255 || hs.node_groups > 255 || cpx > 255 ||
        hs.chunks != cpx * kXcds || hs.blocks != hs.chunks * hs.feature_groups * hs.node_groups ||
        layer > 7 || hs.nodes_per_group > 255 || pc.slices > 255 || hs.copies > 255)
        return hipErrorInvalidValue;
    const uint32_t geo = (uint32_t)d | (uint32_t)hs.feature_groups << 8 |
                         (uint32_t)hs.node_groups << 16 | (uint32_t)cpx << 24;
    const uint32_t mode = (uint32_t)layer | (hs.sibling ? 8u : 0u) | (hs.prefix ? 16u : 0u) |
                          (uint32_t)hs.nodes_per_group << 8 | (uint32_t)pc.slices << 16 |
                          (uint32_t)hs.copies << 24;
    hist_kernel<ROUTED, NP, FPG, SIGNED, MISS><<<hs.blocks, hs.threads, hs.lds_bytes, s>>>(
        xb, w, node_in, ldb, n, hs.chunk_events, hs.xcd_events, geo, mode, pc.cand_gain,
        pc.keys, n_bins, scale, hs.copy_stride, vsign, node_out, pc.rec_f, pc.rec_c,
        pc.rec_g, partial, small, err, tl);
    return hipGetLastError();
}

template <int FPG, bool SIGNED, bool MISS>
hipError_t launch_hist_routed(const HistShape &hs, const uint8_t *xb, int64_t ldb, int64_t n,
                              int d, int n_bins, const uint8_t *node_in, uint8_t *node_out,
                              const float *w, const uint8_t *vsign, const ParentCuts &pc,
                              int layer, int scale, uint64_t *partial, double *small, int *err,
                              unsigned long long *tl, hipStream_t s) {
    const int parents = layer >= 1 ? 1 << (layer - 1) : 0;
#define FBDT_HIST(NPV)                                                                          \
    launch_hist_np<true, NPV, FPG, SIGNED, MISS>(hs, xb, ldb, n, d, n_bins, node_in, node_out, \
                                                 w, vsign, pc, layer, scale, partial, small,   \
                                                 err, tl, s)
    switch (parents) {
    case 0:
    case 1: return FBDT_HIST(1);
    case 2: return FBDT_HIST(2);
    case 4: return FBDT_HIST(4);
    default: return FBDT_HIST(0);
    }
#undef FBDT_HIST
}

template <int FPG>
hipError_t launch_hist_fpg(const HistShape &hs, const uint8_t *xb, int64_t ldb, int64_t n,
                           int d, int n_bins, const uint8_t *node_in, uint8_t *node_out,
                           const float *w, const uint8_t *vsign, const ParentCuts &pc, int layer,
                           bool routed, int scale, uint64_t *partial, double *small, int *err,
                           unsigned long long *tl, hipStream_t s) {
    const ParentCuts none{};
    if (!routed) {
        if (vsign)
            return launch_hist_np<false, 0, FPG, true, false>(hs, xb, ldb, n, d, n_bins, node_in,
                                                              nullptr, w, vsign, none, layer,
                                                              scale, partial, small, err, tl, s);
        return launch_hist_np<false, 0, FPG, false, false>(hs, xb, ldb, n, d, n_bins, node_in,
                                                           nullptr, w, nullptr, none, layer,
                                                           scale, partial, small, err, tl, s);
    }
    // routed passes below the root subtract siblings exactly when no event
    // can stop at a missing value; a fit with missing values histograms both
    // children and takes the stop logic (MISS)
    const bool miss = layer >= 1 && !hs.sibling;
#define FBDT_HIST_R(SG, MS)                                                                     \
    launch_hist_routed<FPG, SG, MS>(hs, xb, ldb, n, d, n_bins, node_in, node_out, w,            \
                                    SG ? vsign : nullptr, pc, layer, scale, partial, small,    \
                                    err, tl, s)
    if (vsign) return miss ? FBDT_HIST_R(true, true) : FBDT_HIST_R(true, false);
    return miss ? FBDT_HIST_R(false, true) : FBDT_HIST_R(false, false);
#undef FBDT_HIST_R
}

hipError_t launch_histogram(const HistShape &hs, const uint8_t *xb, int64_t ldb, int64_t n,
                            int d, int n_bins, const uint8_t *node_in, uint8_t *node_out,
                            const float *w, const uint8_t *vsign, const ParentCuts &pc,
                            int layer, bool routed, int scale, uint64_t *partial, double *small,
                            int *err, hipStream_t s, unsigned long long *tl) {
#define FBDT_HIST_F(F)                                                                          \
    launch_hist_fpg<F>(hs, xb, ldb, n, d, n_bins, node_in, node_out, w, vsign, pc, layer,       \
                       routed, scale, partial, small, err, tl, s)
    switch (hs.features_per_group) {
    case 1: return FBDT_HIST_F(1);
    case 2: return FBDT_HIST_F(2);
    case 4: return FBDT_HIST_F(4);
    case 5: return FBDT_HIST_F(5);
    case 8: return FBDT_HIST_F(8);
    default: return hipErrorInvalidValue;
    }
#undef FBDT_HIST_F
}

hipError_t launch_hist_reference(int kind, const HistShape &hs, const uint8_t *xb, int64_t ldb,
                                 int64_t n, int d, const uint8_t *node, const float *w,
                                 uint32_t *sink, hipStream_t s) {
    hist_reference_kernel<<<hs.blocks, hs.threads, hs.lds_bytes, s>>>(
        kind, xb, ldb, n, d, hs.features_per_group, node, w, hs.feature_groups, hs.node_groups,
        hs.chunks, hs.chunk_events, hs.xcd_events, sink);
    return hipGetLastError();
}

// vs[i] = 1 where v[i] < 0, 0 elsewhere and for the padding [n, npad)
__global__ __launch_bounds__(256) void sign_bytes_kernel(const float *__restrict__ v, int64_t n,
                                                         int64_t npad, uint8_t *__restrict__ vs) {
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < npad;
         i += (int64_t)gridDim.x * blockDim.x)
        vs[i] = (i < n && v[i] < 0.0f) ? 1 : 0;
}

hipError_t launch_sign_bytes(const float *v, int64_t n, int64_t npad, uint8_t *vs, hipStream_t s) {
    sign_bytes_kernel<<<grid_for(npad, 256, 2048), 256, 0, s>>>(v, n, npad, vs);
    return hipGetLastError();
}

hipError_t launch_merge_partials(const uint64_t *partial, int chunks, size_t count, int scale,
                                 const double *small, double *out, hipStream_t s) {
    merge_partials_kernel<<<grid_for((int64_t)count, 256, 2048), 256, 0, s>>>(
        partial, chunks, count, scale, small, out);
    return hipGetLastError();
}

__global__ __launch_bounds__(256) void find_code_kernel(const uint8_t *__restrict__ xb,
                                                        int64_t ldb, int64_t n, uint8_t code,
                                                        int flag, int *__restrict__ err) {
    const int j = blockIdx.y;
    bool found = false;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x)
        found |= xb[(int64_t)j * ldb + i] == code;
    if (__any(found) && threadIdx.x % kWave == 0) atomicOr(err, flag);
}

hipError_t launch_find_code(const uint8_t *xb, int64_t ldb, int64_t n, int d, uint8_t code,
                            int flag, int *err, hipStream_t s) {
    const dim3 grid((unsigned)grid_for(n, 256, 256), (unsigned)d);
    find_code_kernel<<<grid, 256, 0, s>>>(xb, ldb, n, code, flag, err);
    return hipGetLastError();
}

hipError_t launch_abs_sum(const float *w, int64_t n, double *block_partial, double *out,
                          hipStream_t s) {
    abs_sum_kernel<<<kValidateBlocks, 256, 0, s>>>(w, n, block_partial);
    sum_blocks_kernel<<<1, 64, 0, s>>>(block_partial, kValidateBlocks, out);
    return hipGetLastError();
}

int cut_slices(int n_bins) { return (n_bins - 1 + kCutSlice - 1) / kCutSlice; }

hipError_t launch_best_cuts_f64(const double *hist, int n_nodes, int d, int n_bins,
                                double *cand_gain, int *cand_cut, hipStream_t s) {
    best_cuts_f64_kernel<<<n_nodes * d, kWave, 0, s>>>(hist, d, n_bins, cand_gain, cand_cut);
    return hipGetLastError();
}

hipError_t launch_cut_scan(const uint64_t *partial, int chunks, int scale, const double *small,
                           const uint32_t *sany, double *small_next, uint32_t *sany_next,
                           size_t small_next_count, int hnodes, int d,
                           int n_bins, int mode, double *cand_gain, int *cand_cut,
                           const uint64_t *hparent, uint64_t *hout, hipStream_t s,
                           const uint2 *lchunks, uint32_t *clear_words, int clear_count,
                           unsigned long long *keys, unsigned long long *keys_next) {
    const int S = cut_slices(n_bins);
    // one workgroup per (histogrammed node, or parent, feature, slice)
    const int groups = mode == kCutStopped ? hnodes / 2 : hnodes;
    if ((mode == kCutStopped && hnodes % 2 != 0) || (mode != kCutPlain && !hparent))
        return hipErrorInvalidValue;
    if (keys && (mode == kCutPlain ? groups : 2 * groups) > kKeyNodes) return hipErrorInvalidValue;
    // rows padded to a multiple of the XCD count (see the kernel)
    const int blocks = (groups * d + kXcds - 1) / kXcds * kXcds * S;
#define FBDT_CUT(M)                                                                             \
    cut_scan_kernel<M><<<blocks, kCutWaves * kWave, 0, s>>>(                                    \
        partial, chunks, scale, small, small_next, small_next_count, hnodes, d, n_bins, S,      \
        cand_gain, cand_cut, M == kCutPlain ? nullptr : hparent, hout, lchunks, clear_words,     \
        clear_count, sany, sany_next, keys, keys_next)
    switch (mode) {
    case kCutPlain: FBDT_CUT(kCutPlain); break;
    case kCutSibling: FBDT_CUT(kCutSibling); break;
    case kCutStopped: FBDT_CUT(kCutStopped); break;
    default: return hipErrorInvalidValue;
    }
#undef FBDT_CUT
    return hipGetLastError();
}

hipError_t launch_select_cuts(const double *cand_gain, const int *cand_cut, int n_nodes, int d,
                              int slices, uint8_t *out_f, uint8_t *out_c, double *out_g,
                              hipStream_t s) {
    select_cuts_kernel<<<n_nodes, kWave, 0, s>>>(cand_gain, cand_cut, d, slices, out_f, out_c,
                                                 out_g);
    return hipGetLastError();
}

int leaf_blocks(int64_t n, int depth, bool missing, int cu_count) {
    return xcd_grid(n, (int64_t)kLeafE * leaf_threads(depth, missing), cu_count);
}

size_t leaf_lds_bytes(int depth, bool missing) {
    const size_t C = (size_t)leaf_columns(depth, missing);
    const size_t nv = 2 * (size_t)leaf_slots(depth, missing);
    return (nv * (C + 1) + (C >= nv ? C : nv)) * sizeof(double);
}

template <bool ROUTED, int NP>
void leaf_go(int blocks, hipStream_t s, const uint8_t *xb, int64_t ldb, int64_t n, int d,
             const uint8_t *node_in, uint8_t *node_out, const ParentCuts &pc, int depth,
             bool missing, const float *v, const double *yts, double *leaf_partial, int *err) {
    leaf_kernel<ROUTED, NP><<<blocks, leaf_threads(depth, missing), leaf_lds_bytes(depth, missing),
                              s>>>(xb, ldb, n, d, node_in, node_out, pc.cand_gain, pc.keys,
                                   pc.slices, pc.rec_f, pc.rec_c, pc.rec_g, depth, missing, v, yts,
                                   leaf_partial, err, xcd_range(n));
}

hipError_t launch_leaf(const uint8_t *xb, int64_t ldb, int64_t n, int d, const uint8_t *node_in,
                       uint8_t *node_out, const ParentCuts &pc, int depth, bool missing,
                       bool routed, const float *v, const double *yts, int blocks,
                       double *leaf_partial, int *err, hipStream_t s) {
    if (missing && leaf_lds_bytes(depth, missing) > kLeafMaxLds) return hipErrorInvalidValue;
#define FBDT_LEAF(R, NPV, NI, NO, PC)                                                           \
    leaf_go<R, NPV>(blocks, s, xb, ldb, n, d, NI, NO, PC, depth, missing, v, yts, leaf_partial, err)
    if (!routed) {
        FBDT_LEAF(false, 0, node_in, nullptr, ParentCuts{});
    } else {
        switch (1 << (depth - 1)) {   // parents of the leaves
        case 1: FBDT_LEAF(true, 1, node_in, node_out, pc); break;
        case 2: FBDT_LEAF(true, 2, node_in, node_out, pc); break;
        case 4: FBDT_LEAF(true, 4, node_in, node_out, pc); break;
        default: FBDT_LEAF(true, 0, node_in, node_out, pc); break;
        }
    }
#undef FBDT_LEAF
    return hipGetLastError();
}

hipError_t launch_leaf_finalize(const double *leaf_partial, int blocks, int depth, bool missing,
                                double eta, double *leaf_out, hipStream_t s) {
    if (2 * leaf_slots(depth, missing) > kLeafSumSlots) return hipErrorInvalidValue;
    leaf_finalize_kernel<<<1, kLeafReduceThreads, 0, s>>>(
        leaf_partial, blocks, leaf_slots(depth, missing), missing ? (1 << depth) - 1 : 0, eta,
        leaf_out);
    return hipGetLastError();
}

hipError_t launch_route_layer(const uint8_t *xb, int64_t ldb, int64_t n, int d,
                              const uint8_t *node_in, uint8_t *node_out, const ParentCuts &pc,
                              int layer, bool miss, int *err, int cu_count, hipStream_t s) {
    if (layer < 1 || (1 << (layer - 1)) > 64) return hipErrorInvalidValue;
    // two workgroups of 1024 threads per CU (workload 4's leaf routing: 31
    // -> 29.4 us against one; when every workgroup still reduced the
    // parents' candidates itself, one per CU took 34 us against 41 with
    // four workgroups of 256)
    const int64_t R = xcd_range(n);
    int64_t per = (R + (int64_t)kHistE * kRouteLayerThreads - 1) /
                  ((int64_t)kHistE * kRouteLayerThreads);
    const int64_t cap = 2 * cu_count / kXcds > 0 ? 2 * cu_count / kXcds : 1;
    if (per > cap) per = cap;
    if (per < 1) per = 1;
    route_layer_kernel<<<(unsigned)(kXcds * per), kRouteLayerThreads, 0, s>>>(
        xb, ldb, n, d, node_in, node_out, pc.cand_gain, pc.keys, pc.slices, pc.rec_f,
        pc.rec_c, pc.rec_g, layer, miss, err, R);
    return hipGetLastError();
}

bool list_fpg_supported(int f) {
    for (int c : kListFpgSizes)
        if (c == f) return true;
    return false;
}

// The list pass reads the rows of its listed events, about a quarter of
// them, scattered: a row that straddles two 64-byte segments costs both (40
// features in 48-byte rows: 216 MB fetched per layer on workload 4, the
// list pass 57-64 us; in 64-byte rows 53-59 us, the one copy per fit 0.40
// -> 0.62 ms).
int list_row_bytes(int d) {
    int r = 16;
    while (r < d && r < 64) r *= 2;
    return r >= d ? r : (d + 63) & ~63;
}

size_t list_codes_bytes(int64_t n, int d) {
    return (size_t)((n + 255) / 256) * 256 * (size_t)list_row_bytes(d);
}

hipError_t launch_transpose_codes(const uint8_t *xb, int64_t ldb, int64_t n, int d, uint8_t *xr,
                                  hipStream_t s) {
    const int dr = list_row_bytes(d);
    if (d < 1 || dr > 256 || n < 1) return hipErrorInvalidValue;
    // events per workgroup: up to 1024, as many as a 32 KiB tile holds, so
    // that several workgroups share a CU (10M x 40 in 64-byte rows: 0.62 ms
    // with 64 KiB tiles, 0.52 ms with 32 KiB, 0.64 ms with 16 KiB)
    const size_t row = (size_t)(dr / 4 + 1) * 4;
    int E = (int)std::min<size_t>(1024, 32768 / row) & ~63;
    if (E < 64) return hipErrorInvalidValue;
    transpose_codes_kernel<<<(unsigned)((n + E - 1) / E), kTransposeThreads, (size_t)E * row, s>>>(
        xb, ldb, n, d, xr, dr, E);
    return hipGetLastError();
}

ListShape plan_list_histogram(int d, int lists, int cu_count, size_t max_lds, int fpg,
                              int parts, int copies) {
    ListShape ls{};
    // the fewest feature groups whose rows fit the LDS (one row of 256 bins
    // x 2 classes per feature; the kernel has no static LDS), then the
    // smallest built group size that covers d in that many groups
    int f = fpg;
    if (f <= 0) {
        int fmax = kListFpgSizes[0];
        for (int c : kListFpgSizes)
            if ((size_t)c * kRowBytes <= max_lds) fmax = c;
        const int g = (d + fmax - 1) / fmax;
        const int need = (d + g - 1) / g;
        f = fmax;
        for (int c : kListFpgSizes)
            if (c >= need) {
                f = c;
                break;
            }
    }
    ls.fpg = f;
    ls.groups = (d + f - 1) / f;
    ls.lists = lists;
    // about one workgroup per CU (parts per feature group), shared among the
    // lists in proportion to their lengths; more than `lists` of them
    int c = parts > 0 ? parts : cu_count / ls.groups;
    if (c < lists + 1) c = lists + 1;
    ls.parts = c;
    const int total = c * ls.groups;
    ls.per_xcd = (total + kXcds - 1) / kXcds;
    ls.blocks = kXcds * ls.per_xcd;
    const size_t one = (size_t)f * kRowBytes;
    int cp = copies > 0 ? copies : 1;
    while (cp > 1 && (size_t)cp * (one + kHistCopyShift) > max_lds) cp >>= 1;
    ls.copies = cp;
    ls.copy_stride = cp > 1 ? (int)(one + kHistCopyShift) : (int)one;
    ls.lds_bytes = cp > 1 ? (size_t)cp * ls.copy_stride : one;
    return ls;
}

hipError_t launch_route_list(const uint8_t *xb, int64_t ldb, int64_t n, int d, int n_bins,
                             const uint8_t *node_in, uint8_t *node_out, const float *w,
                             const uint8_t *vsign, const ParentCuts &pc, int layer, bool miss,
                             int lmode, const uint64_t *hparent, int scale, const uint32_t *cap_prev,
                             uint32_t cap_root, uint32_t *cursor,
                             uint32_t *lstart, uint32_t *lcap, uint32_t *lside, uint2 *list,
                             double *small, uint32_t *sany, int *err, hipStream_t s) {
    if (layer < 1 || layer > 6 || n < 1 || n > kListMaxEvents) return hipErrorInvalidValue;
    if ((layer == 1) != (node_in == nullptr) || (layer == 1) != (cap_prev == nullptr))
        return hipErrorInvalidValue;
    if ((1 << layer) > kListMaxSlots || (lmode != kCutPlain && !hparent) || lmode < kCutPlain ||
        lmode > kCutStopped)
        return hipErrorInvalidValue;
    const uint32_t tau_bits = (uint32_t)(127 + 23 - scale) << 23;   // 2^(23 - scale)
    if (23 - scale < -126) return hipErrorInvalidValue;
    const int64_t R = xcd_range(n);
    const bool off32 = (uint64_t)d * (uint64_t)ldb <= 0xffffffffull;
    const int64_t E = vsign ? (off32 ? route_list_events<true, true>() : route_list_events<true, false>())
                            : (off32 ? route_list_events<false, true>() : route_list_events<false, false>());
    const unsigned blocks = (unsigned)(kXcds * ((R + E - 1) / E));
#define FBDT_ROUTE_LIST(SG, O32)                                                                \
    route_list_kernel<SG, O32><<<blocks, kRouteListThreads, 0, s>>>(                            \
        xb, ldb, n, d, n_bins, node_in, node_out, w, vsign, pc.cand_gain, pc.keys, pc.slices, \
        pc.rec_f, pc.rec_c, pc.rec_g, layer, miss, lmode, hparent, tau_bits, cap_prev, cap_root,  \
        cursor, lstart, lcap, lside, list, small, err, R, sany)
    if (vsign && off32)
        FBDT_ROUTE_LIST(true, true);
    else if (vsign)
        FBDT_ROUTE_LIST(true, false);
    else if (off32)
        FBDT_ROUTE_LIST(false, true);
    else
        FBDT_ROUTE_LIST(false, false);
#undef FBDT_ROUTE_LIST
    return hipGetLastError();
}

template <int FPG>
void hist_list_go(const ListShape &ls, int lmode, bool signed_w, hipStream_t s, const uint2 *list,
                  const uint32_t *lstart, const uint32_t *lcap, const uint32_t *cursor,
                  const uint32_t *lside, const uint8_t *xr, int dr, int d, int nbins, int scale,
                  uint2 *lchunks, uint64_t *partial, int *err, uint32_t *cnt_out) {
    const bool miss = nbins <= kMissingCode;
    if (signed_w)
        hist_list_kernel<FPG, true><<<ls.blocks, 1024, ls.lds_bytes, s>>>(
            list, lstart, lcap, cursor, lside, xr, dr, d, nbins, miss, ls.groups, ls.parts,
            ls.lists, lmode, ls.per_xcd, scale, ls.copies, ls.copy_stride, lchunks, partial, err,
            cnt_out);
    else
        hist_list_kernel<FPG, false><<<ls.blocks, 1024, ls.lds_bytes, s>>>(
            list, lstart, lcap, cursor, lside, xr, dr, d, nbins, miss, ls.groups, ls.parts,
            ls.lists, lmode, ls.per_xcd, scale, ls.copies, ls.copy_stride, lchunks, partial, err,
            cnt_out);
}

hipError_t launch_hist_list(const ListShape &ls, int lmode, const uint2 *list,
                            const uint32_t *lstart, const uint32_t *lcap, const uint32_t *cursor,
                            const uint32_t *lside, const uint8_t *xr, int d, int n_bins,
                            bool signed_w, int scale, uint2 *lchunks, uint64_t *partial, int *err,
                            uint32_t *cnt_out, hipStream_t s) {
    if (ls.lists < 1 || ls.lists > kListMaxSlots || ls.groups * ls.fpg < d ||
        ls.parts <= ls.lists || ls.blocks != kXcds * ls.per_xcd ||
        ls.per_xcd * kXcds < ls.parts * ls.groups ||
        (ls.copies & (ls.copies - 1)) != 0 || ls.lds_bytes < (size_t)ls.fpg * kRowBytes)
        return hipErrorInvalidValue;
    const int dr = list_row_bytes(d);
    switch (ls.fpg) {
    case 4: hist_list_go<4>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    case 8: hist_list_go<8>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    case 12: hist_list_go<12>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    case 20: hist_list_go<20>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    case 28: hist_list_go<28>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    case 36: hist_list_go<36>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    case 40: hist_list_go<40>(ls, lmode, signed_w, s, list, lstart, lcap, cursor, lside, xr, dr, d, n_bins, scale, lchunks, partial, err, cnt_out); break;
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

hipError_t launch_route(const uint8_t *xb, int64_t ldb, int64_t n, int d, uint8_t *node,
                        const uint8_t *cut_f, const uint8_t *cut_c, int layer, int *err,
                        hipStream_t s) {
    route_kernel<<<grid_for(n, 256, 4096), 256, 0, s>>>(xb, ldb, n, d, node, cut_f, cut_c, layer,
                                                       err);
    return hipGetLastError();
}

ApplyShape plan_apply(int64_t n, int d_used, int n_trees, int depth, bool missing,
                      int cu_count, size_t max_lds, int threads) {
    ApplyShape as{};
    as.d_used = d_used;
    as.missing = missing;
    // boost weights per tree: the leaves, or with missing values every node
    const int nin = (1 << depth) - 1, nleaf = missing ? 2 * nin + 1 : 1 << depth;
    const size_t lds_cap = max_lds > kHistStaticLdsReserve ? max_lds - kHistStaticLdsReserve : 0;
    as.shallow = depth <= kApplyShallowDepth && !missing;
    if (as.shallow) {
        // workgroups of 512 threads (two per CU for 40 features and 400
        // trees of depth 3, measured best); the tile of codes takes at most
        // 96 KiB, the leaf values of as many trees as fit the rest
        int t = threads > 0 ? threads : 512;
        while (t > 64 && (size_t)d_used * (2 * t + 8) > 96 * 1024) t -= 64;
        as.threads = t;
        const size_t xtile = (size_t)d_used * (2 * t + 8);
        const size_t room = lds_cap > xtile + 64 ? lds_cap - xtile - 64 : 0;
        int64_t tpc = (int64_t)(room / ((size_t)nleaf * 8));
        if (tpc < 1) tpc = 1;
        if (tpc > n_trees) tpc = n_trees;
        as.trees_per_chunk = (int)tpc;
        as.lds_bytes = (size_t)tpc * nleaf * 8 + xtile;
    } else {
        // 768 threads (512 for depth 4) measured best on 8M events x 40
        // features: two workgroups per CU keep 24 wavefronts resident
        // (fewer when the tile of codes would pass 96 KiB)
        int t = threads > 0 ? threads : (depth == 4 ? 512 : 768);
        while (t > 64 && (size_t)d_used * (t + 4) > 96 * 1024) t -= 64;
        as.threads = t;
        const size_t xtile = (size_t)d_used * (as.threads + 4);
        const size_t per_tree = (size_t)nleaf * 8 + (size_t)nin * 2;
        size_t budget = 65536;
        if (budget < xtile + per_tree + 64) budget = lds_cap;
        size_t room = budget > xtile + 64 ? budget - xtile - 64 : 0;
        int64_t tpc = (int64_t)(room / per_tree);
        if (tpc < 1) tpc = 1;
        if (tpc > n_trees) tpc = n_trees;
        as.trees_per_chunk = (int)tpc;
        as.lds_bytes =
            (size_t)tpc * nleaf * 8 + ((((size_t)tpc * nin) + 3) & ~(size_t)3) * 2 + xtile;
    }
    const int64_t tile_events = as.shallow ? 2 * (int64_t)as.threads : as.threads;
    const int64_t ntiles = (n + tile_events - 1) / tile_events;
    int64_t blocks = (int64_t)cu_count * (as.shallow ? 4 : 8);
    if (blocks > ntiles) blocks = ntiles;
    if (blocks < 1) blocks = 1;
    as.blocks = (int)blocks;
    return as;
}

hipError_t launch_apply(const ApplyShape &as, const uint8_t *xb, int64_t ldb, int64_t n,
                        const uint16_t *cuts, const uint32_t *nodes, const double *leaves,
                        int n_trees, int depth, double f0, float *prob, double *score,
                        hipStream_t s) {
    if (as.shallow) {
        if (!nodes) return hipErrorInvalidValue;
#define FBDT_APPLY_S(DV)                                                                        \
    apply_shallow_kernel<DV, false><<<as.blocks, as.threads, as.lds_bytes, s>>>(                \
        xb, ldb, nullptr, 0, nullptr, 0, n, as.d_used, nodes, leaves, n_trees,                 \
        as.trees_per_chunk, f0, prob, score)
        switch (depth) {
        case 1: FBDT_APPLY_S(1); break;
        case 2: FBDT_APPLY_S(2); break;
        case 3: FBDT_APPLY_S(3); break;
        default: return hipErrorInvalidValue;
        }
#undef FBDT_APPLY_S
        return hipGetLastError();
    }
    apply_kernel<<<as.blocks, as.threads, as.lds_bytes, s>>>(xb, ldb, n, as.d_used, cuts, leaves,
                                                            n_trees, depth, as.missing,
                                                            as.trees_per_chunk, f0, prob, score);
    return hipGetLastError();
}

ApplyShape plan_importance(int64_t n, int d_used, int n_trees, int depth, bool missing,
                           int cu_count, size_t max_lds) {
    ApplyShape as{};
    as.d_used = d_used;
    as.missing = missing;
    const int nin = (1 << depth) - 1;
    const size_t lds_cap = max_lds > kHistStaticLdsReserve ? max_lds - kHistStaticLdsReserve : 0;
    // one event per thread: its float64 accumulator column and code column
    // take at most 96 KiB over the workgroup, the forest chunk the rest
    int t = 256;
    while (t > 64 && (size_t)d_used * ((size_t)t * 8 + t + 4) > 96 * 1024) t -= 64;
    as.threads = t;
    const size_t fixed = (size_t)d_used * ((size_t)t * 8 + t + 4) + 64;
    const size_t per_tree = (size_t)nin * 10;
    const size_t room = lds_cap > fixed ? lds_cap - fixed : 0;
    int64_t tpc = (int64_t)(room / per_tree);
    if (tpc < 1) tpc = 1;
    if (tpc > n_trees) tpc = n_trees;
    as.trees_per_chunk = (int)tpc;
    as.lds_bytes = (size_t)tpc * nin * 8 + (size_t)d_used * t * 8 +
                   ((((size_t)tpc * nin) + 3) & ~(size_t)3) * 2 + (size_t)d_used * (t + 4);
    const int64_t ntiles = (n + t - 1) / t;
    int64_t blocks = (int64_t)cu_count * 4;
    if (blocks > ntiles) blocks = ntiles;
    if (blocks < 1) blocks = 1;
    as.blocks = (int)blocks;
    return as;
}

hipError_t launch_importance(const ApplyShape &as, const uint8_t *xb, int64_t ldb, int64_t n,
                             const uint16_t *cuts, const double *gains, int n_trees, int depth,
                             double *imp, int64_t ldi, int d_out, hipStream_t s) {
    importance_kernel<<<as.blocks, as.threads, as.lds_bytes, s>>>(
        xb, ldb, n, as.d_used, cuts, gains, n_trees, depth, as.missing, as.trees_per_chunk, imp,
        ldi, d_out);
    return hipGetLastError();
}

ApplyShape plan_apply_float(int64_t n, int d_used, int n_trees, int depth, bool missing,
                            int cu_count, size_t max_lds, int threads, size_t table_bytes) {
    if (depth <= kApplyShallowDepth && !missing) {
        // the binned shallow traversal, its tile staged from the values with
        // the threshold table beside it in LDS
        const size_t tb = (table_bytes + 15) & ~(size_t)15;
        ApplyShape as = plan_apply(n, d_used, n_trees, depth, false, cu_count,
                                   max_lds > tb ? max_lds - tb : 0, threads);
        as.lds_bytes += tb;
        return as;
    }
    ApplyShape as{};
    as.d_used = d_used;
    as.missing = missing;
    as.shallow = false;
    const int nin = (1 << depth) - 1, nleaf = missing ? 2 * nin + 1 : 1 << depth;
    const size_t lds_cap = max_lds > kHistStaticLdsReserve ? max_lds - kHistStaticLdsReserve : 0;
    // one event per thread, 768 threads (measured best on 8M events x 40
    // features at depths 3 and 6): the tile of float32 values takes at most
    // 124 KiB, the leaf values (and records) of as many trees as fit the rest
    int t = threads > 0 ? threads : 768;
    while (t > 64 && (size_t)d_used * t * 4 > 124 * 1024) t -= 64;
    as.threads = t;
    const size_t xtile = (size_t)d_used * t * 4;
    const size_t per_tree = (size_t)nleaf * 8 + (size_t)nin * 8;
    const size_t room = lds_cap > xtile + 64 ? lds_cap - xtile - 64 : 0;
    int64_t tpc = (int64_t)(room / per_tree);
    if (tpc < 1) tpc = 1;
    if (tpc > n_trees) tpc = n_trees;
    as.trees_per_chunk = (int)tpc;
    as.lds_bytes = (size_t)tpc * per_tree + xtile;
    const int64_t ntiles = (n + t - 1) / t;
    int64_t blocks = (int64_t)cu_count * 4;
    if (blocks > ntiles) blocks = ntiles;
    if (blocks < 1) blocks = 1;
    as.blocks = (int)blocks;
    return as;
}

hipError_t launch_apply_float(const ApplyShape &as, const float *x, int64_t ldx, int64_t n,
                              const uint2 *rec, const uint32_t *fnodes, const uint32_t *ftab,
                              int ftab_words, const double *leaves, int n_trees, int depth,
                              double f0, float *prob, double *score, hipStream_t s) {
    if (as.shallow) {
        if (!fnodes || !ftab) return hipErrorInvalidValue;
#define FBDT_APPLY_FS(DV)                                                                       \
    apply_shallow_kernel<DV, true><<<as.blocks, as.threads, as.lds_bytes, s>>>(                 \
        nullptr, 0, x, ldx, ftab, ftab_words, n, as.d_used, fnodes, leaves, n_trees,           \
        as.trees_per_chunk, f0, prob, score)
        switch (depth) {
        case 1: FBDT_APPLY_FS(1); break;
        case 2: FBDT_APPLY_FS(2); break;
        case 3: FBDT_APPLY_FS(3); break;
        default: return hipErrorInvalidValue;
        }
#undef FBDT_APPLY_FS
        return hipGetLastError();
    }
#define FBDT_APPLY_F(DV)                                                                        \
    apply_float_kernel<DV><<<as.blocks, as.threads, as.lds_bytes, s>>>(                         \
        x, ldx, n, as.d_used, rec, leaves, n_trees, as.missing, as.trees_per_chunk, f0, prob,  \
        score)
    switch (depth) {
    case 1: FBDT_APPLY_F(1); break;
    case 2: FBDT_APPLY_F(2); break;
    case 3: FBDT_APPLY_F(3); break;
    case 4: FBDT_APPLY_F(4); break;
    case 5: FBDT_APPLY_F(5); break;
    case 6: FBDT_APPLY_F(6); break;
    case 7: FBDT_APPLY_F(7); break;
    default: return hipErrorInvalidValue;
    }
#undef FBDT_APPLY_F
    return hipGetLastError();
}

hipError_t launch_encode(const float *x, int64_t ldx, int64_t n, int d, const float *bounds,
                         int n_bins, uint8_t *xb, int64_t ldb, int *err, hipStream_t s) {
    dim3 grid(grid_for(n, 256, 1024), d);
    encode_kernel<<<grid, 256, 0, s>>>(x, ldx, n, d, bounds, n_bins, xb, ldb, err);
    return hipGetLastError();
}

}  // namespace fbdt
