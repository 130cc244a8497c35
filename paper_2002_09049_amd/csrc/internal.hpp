// Launch interfaces shared by the kernels' translation units and the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace mpq {

// Brackets one kernel launch with events on its stream while timing is on
// (mpq_timing_enable); otherwise does nothing.
class LaunchTimer {
public:
    LaunchTimer(hipStream_t s, const char *name);
    ~LaunchTimer();
    LaunchTimer(const LaunchTimer &) = delete;
    LaunchTimer &operator=(const LaunchTimer &) = delete;

private:
    hipStream_t s_;
    hipEvent_t start_;
    std::string name_;
};

// Inputs of one greedy fit of a layer (see mpq_fit_layer in mpq.h).
struct FitParams {
    const float *W;      // [C][d]
    int64_t C, d;
    int M;               // 2^(bits-1) - 1
    int P;               // max_points
    const float *grid;   // device [G] multipliers, or nullptr for c_g = g / G
    int G;
    double tol;
    int8_t *codes;       // [C][P][d]
    float *scales;       // [C][P]
    int32_t *counts;     // [C]
    float *err;          // [C][P] or nullptr
};

// Layout of the dense candidate search in one workgroup (kFitThreads threads).
struct FitLayout {
    int lanes;      // threads sharing one element slice (>= 64, a power of two)
    int slices;     // element slices: kFitThreads / lanes
    int chunk;      // candidates evaluated per pass: lanes * kCandPerThread
    int passes;     // ceil(G / chunk)
    int64_t dpad;   // d rounded up to a multiple of 16 * slices (zero padded)
    size_t lds;     // dynamic LDS bytes
};

constexpr int kFitThreads = 256;
constexpr int kCandPerThread = 2;

// Dense search: residual staged in LDS, every (element, candidate) pair
// evaluated in fp32 with fp64 block sums.
FitLayout fit_layout(int64_t d, int G);
hipError_t launch_fit(const FitParams &p, const FitLayout &L, hipStream_t s);

// Histogram search: exact O(d M + G) candidate errors, residual in registers.
// One launch fits the channels of up to kMaxBatchLayers layers whose lengths
// select the same kernel variant (hist_variant); the descriptors travel by
// value in the kernel arguments.
constexpr int64_t kHistMaxDim = 32768;
constexpr int kMaxBatchLayers = 40;

struct HistLayer {
    const float *W;     // [C][d]
    int8_t *codes;      // [C][P][d]
    float *scales;      // [C][P]
    int32_t *counts;    // [C]
    float *err;         // [C][P] or nullptr
    // calibration steps (HistBatch::single) only:
    float *xerr;        // [C][P] output error after each point (written by the error pass)
    const float *ref;   // [C] output error of W itself (relative threshold) or nullptr
    int32_t *list;      // [C] channels that took a point in this step, in any order
    int32_t *nlist;     // [P] their number, per step (zero before the first step)
    // asymmetric codes (reading B2): nullptr, or [C] per-channel offsets
    // (the midpoint of w, written by the fit; the points fit w - offset)
    float *offsets;
    // nullptr, or the output error's D for this layer (tiles of 128 rows by
    // 32 k, row-major inside; see err_item_d_offsets): the fit (not in
    // calibration steps) writes each channel's final residual there in fp32,
    // k past d zero
    float *dres;
    int d;
    int c_begin;        // first workgroup of this layer in the launch
};

struct HistBatch {
    int n_layers;
    int M, P, G;
    const float *grid;  // device multipliers or nullptr (default grid)
    double tol;
    int nlat;           // lattice buckets ((2M-1) G + 1) or 0; set by launch_fit_hist
    // Points already stored per channel (start = s >= 1: only the channels
    // whose count is s take part; their residual is rebuilt from the stored
    // points).  single == 0: the fit runs to its end with the stopping rule
    // on ||r||^2 (tol).  single != 0: one step of the fit on a calibration
    // batch: a channel stops if s >= 1 and xerr[s-1] <= thr (thr = eps * ref,
    // or eps when ref is null), else takes point s + 1 and enters the
    // step's list.
    int start;
    int single;
    double eps;
    // reading A2: each point's scale refitted by least squares for its codes
    int refit;
    // reading F1, Algorithm 2's naive point first.  A fresh fit (start 0,
    // single 0) applies the point (fl32(max|w|) / M, [w / a]_Q), keeps it as
    // the only point when ||r||^2 <= tol ||w||^2, and otherwise restarts from
    // w.  A calibration fit's first step (start 0, single != 0) finds the
    // naive point already stored (count 1, its output error in xerr) and
    // keeps it when xerr <= thr; every other channel restarts from w.
    int gate;
    HistLayer L[kMaxBatchLayers];
};
static_assert(sizeof(HistBatch) <= 4096, "kernel arguments");

size_t fit_hist_lds(int G);
bool fit_hist_supports(int64_t d);
int hist_variant(int64_t d);   // layers with equal variants may share a launch
int hist_variant_count();      // variants are 0 .. hist_variant_count() - 1
bool hist_variant_writes_d(int v);   // the variant's fit fills HistLayer::dres
// Channels of up to kSmallMaxDim weights take the short-channel variants
// (fit_small.hip), one per length d: one wavefront per channel, lanes over
// the candidates, evaluated directly; the same batch descriptors and
// results.  Every layer of a launch has channels of length d.
constexpr int64_t kSmallMaxDim = 16;
hipError_t launch_fit_small(const HistBatch &b, int d, int64_t channels, hipStream_t s);
std::string fit_small_name(int d);
// Name of the histogram kernel that fits channels of length d (default grid
// when default_grid, else a caller's grid), as LaunchTimer records it.
std::string hist_kernel_name(int64_t d, int M, int G, bool default_grid);
hipError_t launch_fit_hist(const HistBatch &b, int variant, int64_t channels, hipStream_t s);
// The paper's own grid (Eq. (11), Def. 1): one workgroup of 256 threads per
// channel, channels of up to kPaperMaxDim weights, the layer descriptors of
// the histogram search (HistLayer; the calibration fields unused).
constexpr int64_t kPaperMaxDim = 8192;
struct PaperBatch {
    int n_layers;
    int M, P;
    double tol;
    double eta;          // the maximal step of Eq. (11)
    HistLayer L[kMaxBatchLayers];
};
static_assert(sizeof(PaperBatch) <= 4096, "kernel arguments");
int paper_variant(int64_t d);        // layers with equal variants may share a launch
size_t paper_lds(int64_t dmax);      // dynamic LDS for channels of up to dmax weights
// Channels longer than kPaperMaxDim (up to kPaperBigMaxDim): the variant
// kPaperBigVariant, whose sorted magnitudes and prefix sums live in a global
// scratch of paper_big_slice(dmax) doubles per workgroup; paper_big_grid
// workgroups take the channels in turn.
constexpr int kPaperBigVariant = 5;
constexpr int64_t kPaperBigMaxDim = 32768;
constexpr int64_t kPaperBigGrid = 1024;
int paper_big_grid(int64_t channels);
size_t paper_big_slice(int64_t dmax);
hipError_t launch_fit_paper_big(const PaperBatch &b, int64_t channels, int64_t dmax, double *scratch,
                                hipStream_t s);
hipError_t launch_fit_paper(const PaperBatch &b, int variant, int64_t channels, int64_t dmax,
                            hipStream_t s);

// Zeroes n int32 (a fill kernel: safe under stream capture).
hipError_t launch_zero_i32(int32_t *p, int64_t n, hipStream_t s);

// Output error of Eq. (12) for a list of layers.
struct ErrLayerIn {
    const float *W;
    const int8_t *codes;
    const float *scales;
    const int32_t *counts;
    const float *X;
    float *err;     // nullptr: no err item for this layer
    float *ref;     // nullptr: no ref for this layer
    int64_t C, d, n;
    // err item restricted to the channels rows[0 .. *nrows) (device, read
    // when the kernels run), err[rows[m] * err_stride] written; rows ==
    // nullptr: every channel, err[k * err_stride] (err_stride 0 means 1)
    const int32_t *rows;
    const int32_t *nrows;
    int64_t err_stride;
    // per-channel offsets (reading B2) subtracted from the err item's D rows,
    // or nullptr
    const float *offsets;
    // clipping candidates (cand != nullptr): the item's D rows are the C * Gc
    // candidate residuals w_k - a_kj [w_k / a_kj]_Q (a_kj = cand[k * Gc + j],
    // codes in [-M, M]); err[k * Gc + j] is written
    const float *cand;
    int Gc, M;
    // err item whose D rows the fit already wrote (at err_item_d): no forming
    int d_ready;
};
// The items (an err item per layer with err, a ref item per layer with ref) go
// in launch groups of up to 1024 (one group for any network here); groups are
// independent and may run side by side, each with its own scratch (whose head
// holds the group's descriptor table).
int err_group_count(const ErrLayerIn *in, int n_in);
size_t err_group_scratch_bytes(const ErrLayerIn *in, int n_in, int group);
double err_group_flop(const ErrLayerIn *in, int n_in, int group);
// The parts of a group's launch: the upload of its descriptor table (small
// kernels that depend on nothing the fit writes) and the form, GEMM and
// finish kernels; a caller may enqueue the uploads earlier, beside other work.
constexpr int kErrUpload = 1, kErrKernels = 2;
hipError_t launch_output_error_group(const ErrLayerIn *in, int n_in, int group, int P, void *scratch,
                                     hipStream_t s,
                                     int parts = kErrUpload | kErrKernels);
// Where the err item of in[i] keeps its rows of D (fp32 tiles [ceil(C / 128)]
// [ceil(d / 32)][128][32], row-major inside, k past d zero): for each
// in[i], the byte offset inside its group's scratch in off[i] and the group
// in group[i]; -1 for both when in[i] has no err item or its rows are
// clipping candidates.  Every group's layout is formed once.
void err_item_d_offsets(const ErrLayerIn *in, int n_in, int64_t *off, int *group);

// Clipping of Eq. (13) as the first point: candidate scales, then (after the
// output error of the candidates) the choice of point 1.  One workgroup per
// channel; up to kMaxClipLayers layers per launch.
struct ClipLayer {
    const float *W;        // [C][d]
    float *cand;           // [C][Gc] candidate scales
    const float *ecand;    // [C][Gc] their output errors
    int8_t *codes;         // [C][P][d]
    float *scales;         // [C][P]
    int32_t *counts;       // [C]
    float *err;            // [C][P] or nullptr
    float *xerr;           // [C][P] or nullptr (calibration rule: e_1)
    int d;
    int c_begin;           // first workgroup of this layer
};
constexpr int kMaxClipLayers = 48;
struct ClipBatch {
    int n_layers;
    int M, P, Gc;
    ClipLayer L[kMaxClipLayers];
};
static_assert(sizeof(ClipBatch) <= 4096, "kernel arguments");
hipError_t launch_clip(const ClipBatch &b, int64_t channels, bool choose, hipStream_t s);

// Stream-ordered scratch from a library-owned memory pool of the current
// device (kept, not returned to the system, between calls).
hipError_t scratch_alloc(void **p, size_t bytes, hipStream_t s);
hipError_t scratch_free(void *p, hipStream_t s);

// Reconstruction of Eq. (4) for a list of layers.
struct RecLayer {
    const int8_t *codes;
    const float *scales;
    const int32_t *counts;
    float *W_hat;
    int64_t C, d;
    const float *offsets;   // reading B2: added first, or nullptr
};
constexpr int kMaxRecLayers = 56;
hipError_t launch_reconstruct(const RecLayer *in, int n_in, int P, hipStream_t s);

// Deployment arithmetic (Sec. 3.4).
hipError_t launch_integer_scales(const float *scales, const int32_t *counts, int64_t C, int P, int p,
                                 int32_t *A, unsigned long long *clamped, hipStream_t s);

// Integer forward of up to kMaxIntLayers layers of one load mode in one
// launch (one workgroup per tile of 32 channels by 128 columns); ntm, ntn
// and block_begin are set by launch_int_forward.  Each layer's codes and X
// are below 2^31 bytes.
struct IntLayer {
    const int8_t *codes;    // [C][P][d]
    const int32_t *A;       // [C][P]
    const int32_t *counts;  // [C]
    const int8_t *X;        // [N][d]
    int64_t *Y;             // [C][N]
    int64_t C, d, N;
    int ntm, ntn, block_begin;
};
constexpr int kMaxIntLayers = 32;
struct IntGroup {
    int n_layers;
    int P, p;
    IntLayer L[kMaxIntLayers];
};
static_assert(sizeof(IntGroup) <= 4096, "kernel arguments");
// The operand load width a layer takes (0: 16 bytes, 1: 4 bytes, 2: bytes);
// the layers of one launch share it.
constexpr int kIntModes = 3;
int int_forward_mode(const IntLayer &L);
hipError_t launch_int_forward(IntGroup &g, int mode, hipStream_t s);

}  // namespace mpq
