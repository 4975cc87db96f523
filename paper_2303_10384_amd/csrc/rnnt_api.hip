// C-ABI of the RNN-T / W-Transducer loss library (declarations and contract in
// include/rnnt_mi355x.h).  Host side: argument checks that need no device,
// workspace carve-up, kernel selection and launches on the caller's stream.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cstdint>
#include <mutex>

#include "rnnt_mi355x.h"
#include "rnnt_launch.h"

// Workspace of rnnt_loss_noalloc: one copy on every GPU the library runs on.  In
// host code this name is only a stand-in for the array; its device address is
// looked up per GPU (noalloc_scratch below) and only that address is used.
static __device__ __align__(256) unsigned char scratch[RNNT_NOALLOC_SCRATCH_BYTES];

namespace rnnt {
namespace {

constexpr int kMaxUnits1 = 2048;  // widest U_max + 1 of the grid sweeps (one wavefront, 32 units per lane)

size_t align256(size_t x) { return (x + 255) & ~static_cast<size_t>(255); }

bool dtype_known(int dt) { return dt == RNNT_DTYPE_F32 || dt == RNNT_DTYPE_BF16 || dt == RNNT_DTYPE_F16; }

bool variant_known(int v) {
  return v == RNNT_VARIANT_RNNT || v == RNNT_VARIANT_WRNNT || v == RNNT_VARIANT_WRNNT_ALLOW_IGNORE;
}

rnnt_status_t check_shape(const rnnt_shape_t& s) {
  if (s.B < 1 || s.T_max < 1 || s.U_max < 0 || s.V < 2) return RNNT_ERR_BAD_SHAPE;
  // keep every 32-bit block count and per-utterance row count in range
  const int64_t rows_per_utt = static_cast<int64_t>(s.T_max) * (s.U_max + 1);
  if (rows_per_utt > (int64_t{1} << 30)) return RNNT_ERR_BAD_SHAPE;
  if (static_cast<int64_t>(s.B) * rows_per_utt > (int64_t{1} << 40)) return RNNT_ERR_BAD_SHAPE;
  if (s.V > (1 << 30)) return RNNT_ERR_BAD_SHAPE;
  if (!dtype_known(s.dtype)) return RNNT_ERR_BAD_DTYPE;
  if (s.grad_dtype != s.dtype && s.grad_dtype != RNNT_DTYPE_F32) return RNNT_ERR_BAD_DTYPE;
  return RNNT_OK;
}

// Workspace, all pieces 256-byte aligned (C = B * T_max * (U_max+1) lattice
// cells, one per logits row; S = B * (T_max+U_max+1) * u_pad score cells, u_pad =
// 64 * units per lane of the lattice sweep):
//   rowinfo  B*T_max*(U_max+1) RowInfo        (rnnt_loss)
//   lp2      C double2 {lp_blank, lp_label}, lse2f in their low bits  (rnnt_loss)
//   alpha    S double
//   beta     S double
//   lnp      2*B double
//   status   B int32
struct Layout {
  size_t rowinfo, lp2, alpha, beta, lnp, status, total;
};

Layout make_layout(const rnnt_shape_t& s, bool with_populate) {
  const size_t U1 = static_cast<size_t>(s.U_max) + 1;
  const size_t rows = static_cast<size_t>(s.B) * s.T_max * U1;
  const size_t cells = static_cast<size_t>(s.B) * s.T_max * U1;
  const size_t u_pad = 64 * static_cast<size_t>(units_per_lane(s.U_max + 1));
  const size_t score_cells = static_cast<size_t>(s.B) * (s.T_max + s.U_max + 1) * u_pad;
  Layout L{};
  size_t o = 0;
  if (with_populate) {
    L.rowinfo = o;
    o = align256(o + rows * sizeof(RowInfo));
    L.lp2 = o;
    o = align256(o + cells * 2 * sizeof(double));
  }
  L.alpha = o;
  o = align256(o + score_cells * sizeof(double));
  L.beta = o;
  o = align256(o + score_cells * sizeof(double));
  L.lnp = o;
  o = align256(o + 2 * static_cast<size_t>(s.B) * sizeof(double));
  L.status = o;
  o = align256(o + static_cast<size_t>(s.B) * sizeof(int32_t));
  L.total = o;
  return L;
}

// Workspace of the forced alignment: the lattice form (lp2) as in the loss,
// the decision words B * (T_max+U_max+1) * K uint64, 256-byte aligned pieces.
struct ViterbiLayout {
  size_t lp2, decisions, total;
};

ViterbiLayout make_viterbi_layout(const rnnt_shape_t& s) {
  const size_t U1 = static_cast<size_t>(s.U_max) + 1;
  const size_t cells = static_cast<size_t>(s.B) * s.T_max * U1;
  const size_t words = static_cast<size_t>(s.B) * (s.T_max + s.U_max + 1) * units_per_lane(s.U_max + 1);
  ViterbiLayout L{};
  size_t o = 0;
  L.lp2 = o;
  o = align256(o + cells * 2 * sizeof(double));
  L.decisions = o;
  o = align256(o + words * sizeof(uint64_t));
  L.total = o;
  return L;
}

bool aligned16(const void* ptr) { return (reinterpret_cast<uintptr_t>(ptr) & 15u) == 0; }

// Stream-ordered workspace when the caller passes none.
struct OwnedWorkspace {
  void* ptr = nullptr;
  hipStream_t stream = nullptr;
  ~OwnedWorkspace() {
    if (ptr) (void)hipFreeAsync(ptr, stream);
  }
};

rnnt_status_t take_workspace(void* workspace, size_t workspace_bytes, size_t need, hipStream_t stream,
                             OwnedWorkspace& owned, char** ws) {
  if (workspace && workspace_bytes < need) return RNNT_ERR_WORKSPACE;
  if (workspace && (reinterpret_cast<uintptr_t>(workspace) & 255u)) return RNNT_ERR_ALIGNMENT;
  *ws = static_cast<char*>(workspace);
  if (!*ws) {
    if (hipMallocAsync(&owned.ptr, need, stream) != hipSuccess) return RNNT_ERR_HIP;
    owned.stream = stream;
    *ws = static_cast<char*>(owned.ptr);
  }
  return RNNT_OK;
}

// ---- arc-list lattices -------------------------------------------------------

// Workspace of rnnt_arc_loss, 256-byte aligned pieces (R logits rows, A arcs,
// S states of the plan):
//   lse2     R double   lse2f = log2 sum_v 2^(z_v kLog2eF) per row
//   rec0/1   A0, A1 x 12 bytes  slot records (weight, source LDS slot) of the two sweeps
//   val0/1   S double   forward / backward scores
//   lnp      2*B double
//   status   B int32
//   bad      B int32    bad-data flags of the populate kernel
//   rowinfo  R RowInfo  (with a gradient)
//   occ      A0 x 8 bytes  {posterior, label} per graph-0 slot (with a gradient)
struct ArcLayout {
  size_t lse2, w0, w1, val0, val1, lnp, status, bad, rowinfo, occ, total;
};

ArcLayout make_arc_layout(const rnnt_arc_plan_t& pl) {
  const size_t R = static_cast<size_t>(pl.B) * pl.T_max * (static_cast<size_t>(pl.U_max) + 1);
  const size_t A0 = static_cast<size_t>(pl.num_slots[0]), A1 = static_cast<size_t>(pl.num_slots[1]);
  const size_t S = static_cast<size_t>(pl.num_states);
  ArcLayout L{};
  size_t o = 0;
  L.lse2 = o;
  o = align256(o + R * sizeof(double));
  L.w0 = o;
  o = align256(o + A0 * kSlotWords * sizeof(int32_t));
  L.w1 = o;
  o = align256(o + A1 * kSlotWords * sizeof(int32_t));
  L.val0 = o;
  o = align256(o + S * sizeof(double));
  L.val1 = o;
  o = align256(o + S * sizeof(double));
  L.lnp = o;
  o = align256(o + 2 * static_cast<size_t>(pl.B) * sizeof(double));
  L.status = o;
  o = align256(o + static_cast<size_t>(pl.B) * sizeof(int32_t));
  L.bad = o;
  o = align256(o + static_cast<size_t>(pl.B) * sizeof(int32_t));
  L.rowinfo = o;
  o = align256(o + R * sizeof(RowInfo));
  L.occ = o;
  o = align256(o + A0 * sizeof(int2));
  L.total = o;
  return L;
}

// The descriptor must describe an image of this shape with its arrays in order.
bool plan_consistent(const rnnt_arc_plan_t& pl, const rnnt_shape_t& s) {
  if (pl.B != s.B || pl.T_max != s.T_max || pl.U_max != s.U_max || pl.V != s.V) return false;
  if (pl.num_states < pl.B || pl.num_arcs < 0 || pl.num_levels < pl.B || pl.num_row_arcs < 0 ||
      pl.num_extra_rows < 0 || pl.num_slots[0] < pl.num_arcs || pl.num_slots[1] < pl.num_arcs)
    return false;
  const int64_t R = static_cast<int64_t>(pl.B) * pl.T_max * (static_cast<int64_t>(pl.U_max) + 1);
  if (R >= 0x7fffffffLL || pl.blank < 0 || pl.blank >= pl.V) return false;
  for (int i = 0; i < kImgCount; ++i) {
    if (pl.off[i] < 0 || (pl.off[i] & 255) || pl.off[i] > pl.image_bytes) return false;
    if (i > 0 && pl.off[i] < pl.off[i - 1]) return false;
  }
  return true;
}

// The sweeps take U_max + 1 <= kMaxUnits1 and address an utterance's score rows
// ((T_max + U_max + 1) rows of 64 K float64) through one buffer with 32-bit
// offsets.
bool scores_fit(const rnnt_shape_t& s) {
  return s.U_max + 1 <= kMaxUnits1 &&
         static_cast<int64_t>(s.T_max + s.U_max + 1) * 64 * units_per_lane(s.U_max + 1) * 8 < (int64_t{1} << 31);
}

// ... and read its lattice form (T_max x (U_max+1) cells of 16 bytes) the same way.
bool sweep_fits(const rnnt_shape_t& s) {
  return scores_fit(s) && static_cast<int64_t>(s.T_max) * (s.U_max + 1) * 16 < (int64_t{1} << 31);
}

// Checks of rnnt_loss's arguments that need no device.
rnnt_status_t check_loss_args(const void* logits, const rnnt_shape_t& shape, const int32_t* labels,
                              const int32_t* logit_lens, const int32_t* label_lens, int32_t blank, int variant,
                              const float* loss_out, const void* grad_out) {
  const rnnt_status_t st = check_shape(shape);
  if (st != RNNT_OK) return st;
  if (!logits || !logit_lens || !label_lens || !loss_out || (!labels && shape.U_max > 0))
    return RNNT_ERR_NULL_PTR;
  if (blank < 0 || blank >= shape.V) return RNNT_ERR_BAD_BLANK;
  if (!variant_known(variant)) return RNNT_ERR_BAD_VARIANT;
  if (!aligned16(logits) || (grad_out && !aligned16(grad_out))) return RNNT_ERR_ALIGNMENT;
  if (!sweep_fits(shape)) return RNNT_ERR_UNSUPPORTED;
  return RNNT_OK;
}

// Device address of `scratch` on each GPU, looked up once per GPU with that GPU
// current and kept until the process ends.
constexpr int kMaxDevices = 256;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

rnnt_status_t noalloc_scratch(hipStream_t stream, void** out) {
  int dev = 0;
  if (stream == nullptr) {
    if (hipGetDevice(&dev) != hipSuccess) return RNNT_ERR_HIP;
  } else if (hipStreamGetDevice(stream, &dev) != hipSuccess) {
    return RNNT_ERR_HIP;
  }
  if (dev < 0 || dev >= kMaxDevices) return RNNT_ERR_HIP;
  void* ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (ptr == nullptr) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    ptr = g_scratch[dev].load(std::memory_order_relaxed);
    if (ptr == nullptr) {
      int cur = 0;
      if (hipGetDevice(&cur) != hipSuccess) return RNNT_ERR_HIP;
      if (cur != dev && hipSetDevice(dev) != hipSuccess) return RNNT_ERR_HIP;
      const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
      const hipError_t e_back = (cur != dev) ? hipSetDevice(cur) : hipSuccess;
      if (e != hipSuccess || e_back != hipSuccess || ptr == nullptr) return RNNT_ERR_HIP;
      if (reinterpret_cast<uintptr_t>(ptr) & 255u) return RNNT_ERR_HIP;
      g_scratch[dev].store(ptr, std::memory_order_release);
    }
  }
  *out = ptr;
  return RNNT_OK;
}

}  // namespace
}  // namespace rnnt

using namespace rnnt;

extern "C" {

const char* rnnt_status_string(rnnt_status_t status) {
  switch (status) {
    case RNNT_OK: return "ok";
    case RNNT_ERR_NULL_PTR: return "a required pointer is NULL";
    case RNNT_ERR_BAD_SHAPE: return "bad shape (need B >= 1, T_max >= 1, U_max >= 0, V >= 2, sizes in range)";
    case RNNT_ERR_BAD_BLANK: return "blank outside [0, V)";
    case RNNT_ERR_BAD_DTYPE: return "unknown dtype, or grad_dtype neither dtype nor F32";
    case RNNT_ERR_BAD_VARIANT: return "unknown variant";
    case RNNT_ERR_WORKSPACE: return "workspace smaller than required";
    case RNNT_ERR_ALIGNMENT: return "logits / grad must be 16-byte aligned, workspace 256-byte aligned";
    case RNNT_ERR_HIP: return "HIP runtime error";
    case RNNT_ERR_UNSUPPORTED:
      return "unsupported shape (U_max + 1 > 2048, T_max * (U_max + 1) >= 2^27, or a lattice past the sweep's limits)";
    case RNNT_ERR_BAD_LATTICE: return "arc list breaks the numbering rules, or the plan does not match the call";
    case RNNT_ERR_SCRATCH:
      return "the shape needs more workspace than the static scratch of rnnt_loss_noalloc (RNNT_NOALLOC_SCRATCH_BYTES)";
  }
  return "unknown status";
}

const char* rnnt_version(void) { return "rnnt_mi355x 0.3.0 gfx950"; }

size_t rnnt_loss_workspace_bytes(rnnt_shape_t shape) {
  if (check_shape(shape) != RNNT_OK) return 0;
  return make_layout(shape, true).total;
}

size_t rnnt_lattice_workspace_bytes(rnnt_shape_t shape) {
  rnnt_shape_t s = shape;
  s.dtype = RNNT_DTYPE_F32;
  s.grad_dtype = RNNT_DTYPE_F32;
  if (check_shape(s) != RNNT_OK) return 0;
  return make_layout(s, false).total;
}

rnnt_status_t rnnt_loss_timed(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                              const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                              rnnt_variant_t variant, float* loss_out, void* grad_out, void* workspace,
                              size_t workspace_bytes, hipStream_t stream, hipEvent_t* events) {
  rnnt_status_t st = check_loss_args(logits, shape, labels, logit_lens, label_lens, blank, variant, loss_out,
                                     grad_out);
  if (st != RNNT_OK) return st;
  const Layout L = make_layout(shape, true);
  OwnedWorkspace owned;
  char* ws = nullptr;
  st = take_workspace(workspace, workspace_bytes, L.total, stream, owned, &ws);
  if (st != RNNT_OK) return st;

  const int64_t U1 = shape.U_max + 1;
  const int64_t n_rows = static_cast<int64_t>(shape.B) * shape.T_max * U1;
  const int64_t n_elem = n_rows * shape.V;
  const bool need_grad = grad_out != nullptr;
  auto mark = [&](int i) { return events ? hipEventRecord(events[i], stream) : hipSuccess; };
  if (mark(0) != hipSuccess) return RNNT_ERR_HIP;

  // kernel 1: lse and arc weights in the lattice form
  PopulateParams p1{};
  p1.logits = logits;
  p1.B = shape.B;
  p1.T_max = shape.T_max;
  p1.U_max = shape.U_max;
  p1.V = shape.V;
  p1.blank = blank;
  p1.labels = labels;
  p1.logit_lens = logit_lens;
  p1.label_lens = label_lens;
  p1.n_elem = n_elem;
  p1.lp2 = reinterpret_cast<double2*>(ws + L.lp2);
  p1.pack_lse2f = 1;  // the posterior kernel reads lse2f from the weights
  if (launch_populate_lattice(shape.dtype, p1, stream) != hipSuccess) return RNNT_ERR_HIP;
  if (mark(1) != hipSuccess) return RNNT_ERR_HIP;

  // kernel 2: forward / backward sweeps
  LatticeParams p2{};
  p2.B = shape.B;
  p2.T_max = shape.T_max;
  p2.U_max = shape.U_max;
  p2.V = shape.V;
  p2.blank = blank;
  p2.labels = labels;
  p2.logit_lens = logit_lens;
  p2.label_lens = label_lens;
  p2.lp2 = p1.lp2;
  p2.alpha = reinterpret_cast<double*>(ws + L.alpha);
  p2.beta = reinterpret_cast<double*>(ws + L.beta);
  p2.u_pad = 64 * units_per_lane(shape.U_max + 1);
  p2.lnp2_fwd = reinterpret_cast<double*>(ws + L.lnp);
  p2.lnp2_bwd = p2.lnp2_fwd + shape.B;
  p2.status = reinterpret_cast<int32_t*>(ws + L.status);
  p2.loss_f32 = loss_out;
  const hipError_t e2 = need_grad ? launch_lattice_scores(variant, p2, stream) : launch_lattice_loss_only(variant, p2, stream);
  if (e2 != hipSuccess) return RNNT_ERR_HIP;
  if (mark(2) != hipSuccess) return RNNT_ERR_HIP;

  if (need_grad) {
    // kernel 2b: arc posteriors -> row records
    PostParams pb{};
    pb.B = shape.B;
    pb.T_max = shape.T_max;
    pb.U_max = shape.U_max;
    pb.labels = labels;
    pb.logit_lens = logit_lens;
    pb.label_lens = label_lens;
    pb.status = p2.status;
    pb.lp2 = p1.lp2;
    pb.alpha = p2.alpha;
    pb.beta = p2.beta;
    pb.u_pad = p2.u_pad;
    pb.lnp2_fwd = p2.lnp2_fwd;
    pb.lnp2_bwd = p2.lnp2_bwd;
    pb.n_rows = n_rows;
    pb.rowinfo = reinterpret_cast<RowInfo*>(ws + L.rowinfo);
    if (launch_posteriors_rows(pb, stream) != hipSuccess) return RNNT_ERR_HIP;
  }
  if (mark(3) != hipSuccess) return RNNT_ERR_HIP;

  if (need_grad) {
    // kernel 3: gradient
    GradParams p3{};
    p3.logits = logits;
    p3.grad = grad_out;
    p3.rowinfo = reinterpret_cast<RowInfo*>(ws + L.rowinfo);
    p3.n_elem = n_elem;
    p3.n_rows = n_rows;
    p3.V = shape.V;
    p3.blank = blank;
    if (launch_grad(shape.dtype, shape.grad_dtype, p3, stream) != hipSuccess) return RNNT_ERR_HIP;
  }
  if (mark(4) != hipSuccess) return RNNT_ERR_HIP;
  return RNNT_OK;
}

rnnt_status_t rnnt_loss(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                        const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                        rnnt_variant_t variant, float* loss_out, void* grad_out, void* workspace,
                        size_t workspace_bytes, hipStream_t stream) {
  return rnnt_loss_timed(logits, shape, labels, logit_lens, label_lens, blank, variant, loss_out, grad_out,
                         workspace, workspace_bytes, stream, nullptr);
}

rnnt_status_t rnnt_loss_noalloc(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                                const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                                rnnt_variant_t variant, float* loss_out, void* grad_out, hipStream_t stream) {
  // every host check first: argument errors and a shape too large for the
  // scratch return before any HIP call
  const rnnt_status_t st = check_loss_args(logits, shape, labels, logit_lens, label_lens, blank, variant, loss_out,
                                           grad_out);
  if (st != RNNT_OK) return st;
  const size_t need = make_layout(shape, true).total;
  if (need > RNNT_NOALLOC_SCRATCH_BYTES) return RNNT_ERR_SCRATCH;
  void* ws = nullptr;
  const rnnt_status_t sst = noalloc_scratch(stream, &ws);
  if (sst != RNNT_OK) return sst;
  // a non-null workspace of sufficient size: rnnt_loss_timed allocates nothing
  return rnnt_loss_timed(logits, shape, labels, logit_lens, label_lens, blank, variant, loss_out, grad_out, ws,
                         RNNT_NOALLOC_SCRATCH_BYTES, stream, nullptr);
}

size_t rnnt_viterbi_workspace_bytes(rnnt_shape_t shape) {
  rnnt_shape_t s = shape;
  s.grad_dtype = s.dtype;
  if (check_shape(s) != RNNT_OK) return 0;
  return make_viterbi_layout(s).total;
}

rnnt_status_t rnnt_viterbi_timed(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                                 const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                                 rnnt_variant_t variant, float* score_out, int32_t* label_frames_out,
                                 int32_t* span_out, void* workspace, size_t workspace_bytes, hipStream_t stream,
                                 hipEvent_t* events) {
  shape.grad_dtype = shape.dtype;  // no gradient here
  rnnt_status_t st = check_shape(shape);
  if (st != RNNT_OK) return st;
  if (!logits || !logit_lens || !label_lens || !score_out || (!labels && shape.U_max > 0) ||
      (!label_frames_out && shape.U_max > 0))
    return RNNT_ERR_NULL_PTR;
  if (blank < 0 || blank >= shape.V) return RNNT_ERR_BAD_BLANK;
  if (!variant_known(variant)) return RNNT_ERR_BAD_VARIANT;
  if (!aligned16(logits)) return RNNT_ERR_ALIGNMENT;
  if (!sweep_fits(shape)) return RNNT_ERR_UNSUPPORTED;
  const ViterbiLayout L = make_viterbi_layout(shape);
  OwnedWorkspace owned;
  char* ws = nullptr;
  st = take_workspace(workspace, workspace_bytes, L.total, stream, owned, &ws);
  if (st != RNNT_OK) return st;
  auto mark = [&](int i) { return events ? hipEventRecord(events[i], stream) : hipSuccess; };
  if (mark(0) != hipSuccess) return RNNT_ERR_HIP;

  PopulateParams p1{};
  p1.logits = logits;
  p1.B = shape.B;
  p1.T_max = shape.T_max;
  p1.U_max = shape.U_max;
  p1.V = shape.V;
  p1.blank = blank;
  p1.labels = labels;
  p1.logit_lens = logit_lens;
  p1.label_lens = label_lens;
  p1.n_elem = static_cast<int64_t>(shape.B) * shape.T_max * (shape.U_max + 1) * shape.V;
  p1.lp2 = reinterpret_cast<double2*>(ws + L.lp2);
  p1.pack_lse2f = 0;  // the alignment's ties stay exact in the unmodified weights
  if (launch_populate_lattice(shape.dtype, p1, stream) != hipSuccess) return RNNT_ERR_HIP;
  if (mark(1) != hipSuccess) return RNNT_ERR_HIP;

  ViterbiParams pv{};
  pv.B = shape.B;
  pv.T_max = shape.T_max;
  pv.U_max = shape.U_max;
  pv.V = shape.V;
  pv.blank = blank;
  pv.labels = labels;
  pv.logit_lens = logit_lens;
  pv.label_lens = label_lens;
  pv.lp2 = p1.lp2;
  pv.decisions = reinterpret_cast<uint64_t*>(ws + L.decisions);
  pv.score_out = score_out;
  pv.label_frames = label_frames_out;
  pv.span = span_out;
  if (launch_viterbi(variant, pv, stream) != hipSuccess) return RNNT_ERR_HIP;
  return mark(2) == hipSuccess ? RNNT_OK : RNNT_ERR_HIP;
}

rnnt_status_t rnnt_viterbi(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                           const int32_t* logit_lens, const int32_t* label_lens, int32_t blank,
                           rnnt_variant_t variant, float* score_out, int32_t* label_frames_out, int32_t* span_out,
                           void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return rnnt_viterbi_timed(logits, shape, labels, logit_lens, label_lens, blank, variant, score_out,
                            label_frames_out, span_out, workspace, workspace_bytes, stream, nullptr);
}

size_t rnnt_arc_loss_workspace_bytes(const rnnt_arc_plan_t* plan) {
  if (!plan) return 0;
  return make_arc_layout(*plan).total;
}

rnnt_status_t rnnt_arc_loss_timed(const void* logits, rnnt_shape_t shape, const int32_t* logit_lens,
                                  const int32_t* label_lens, const rnnt_arc_plan_t* plan, const void* plan_image,
                                  float* loss_out, void* grad_out, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream, hipEvent_t* events) {
  rnnt_status_t st = check_shape(shape);
  if (st != RNNT_OK) return st;
  if (!logits || !logit_lens || !label_lens || !plan || !plan_image || !loss_out) return RNNT_ERR_NULL_PTR;
  if (!plan_consistent(*plan, shape)) return RNNT_ERR_BAD_LATTICE;
  if (!aligned16(logits) || (grad_out && !aligned16(grad_out)) || !aligned16(plan_image))
    return RNNT_ERR_ALIGNMENT;
  const ArcLayout L = make_arc_layout(*plan);
  OwnedWorkspace owned;
  char* ws = nullptr;
  st = take_workspace(workspace, workspace_bytes, L.total, stream, owned, &ws);
  if (st != RNNT_OK) return st;
  const char* img = static_cast<const char*>(plan_image);
  auto arr = [&](int i) { return img + plan->off[i]; };

  const int64_t U1 = shape.U_max + 1;
  const int64_t n_rows = static_cast<int64_t>(shape.B) * shape.T_max * U1;
  auto mark = [&](int i) { return events ? hipEventRecord(events[i], stream) : hipSuccess; };
  if (mark(0) != hipSuccess) return RNNT_ERR_HIP;

  // kernel 1 (rows form): lse2f of every valid row
  PopulateParams p1{};
  p1.logits = logits;
  p1.B = shape.B;
  p1.T_max = shape.T_max;
  p1.U_max = shape.U_max;
  p1.V = shape.V;
  p1.blank = plan->blank;
  p1.labels = nullptr;
  p1.logit_lens = logit_lens;
  p1.label_lens = label_lens;
  p1.n_elem = n_rows * shape.V;
  p1.lse2_rows = reinterpret_cast<double*>(ws + L.lse2);
  p1.clear_flags = reinterpret_cast<int32_t*>(ws + L.bad);
  if (launch_populate_rows(shape.dtype, p1, stream) != hipSuccess) return RNNT_ERR_HIP;
  if (mark(1) != hipSuccess) return RNNT_ERR_HIP;

  // arc weights in both sweep orders
  ArcPopulateParams pp{};
  pp.logits = logits;
  pp.B = shape.B;
  pp.T_max = shape.T_max;
  pp.U_max = shape.U_max;
  pp.V = shape.V;
  pp.n_slots0 = plan->num_slots[0];
  pp.n_slots1 = plan->num_slots[1];
  pp.n_rows = static_cast<int32_t>(n_rows);
  pp.logit_lens = logit_lens;
  pp.label_lens = label_lens;
  pp.arcs = reinterpret_cast<const int4*>(arr(kImgArcs));
  pp.score = reinterpret_cast<const float*>(arr(kImgScore));
  pp.perm = reinterpret_cast<const int32_t*>(arr(kImgPerm));
  pp.loc0 = reinterpret_cast<const int32_t*>(arr(kImgLoc0));
  pp.loc1 = reinterpret_cast<const int32_t*>(arr(kImgLoc1));
  pp.lse2_rows = p1.lse2_rows;
  pp.bad = p1.clear_flags;
  pp.rec0 = reinterpret_cast<int32_t*>(ws + L.w0);
  pp.rec1 = reinterpret_cast<int32_t*>(ws + L.w1);
  if (launch_arc_weights(shape.dtype, pp, stream) != hipSuccess) return RNNT_ERR_HIP;
  if (mark(2) != hipSuccess) return RNNT_ERR_HIP;

  // forward and backward sweeps
  ArcSweepParams ps{};
  ps.B = shape.B;
  ps.T_max = shape.T_max;
  ps.U_max = shape.U_max;
  ps.logit_lens = logit_lens;
  ps.label_lens = label_lens;
  ps.utt = reinterpret_cast<const int4*>(arr(kImgUtt));
  ps.ends = reinterpret_cast<const int4*>(arr(kImgEnds));
  ps.slots = reinterpret_cast<const int4*>(arr(kImgSlots));
  for (int g = 0; g < 2; ++g) {
    ps.level[g] = reinterpret_cast<const int4*>(arr(g ? kImgLevel1 : kImgLevel0));
    ps.seg[g] = reinterpret_cast<const int32_t*>(arr(g ? kImgSeg1 : kImgSeg0));
    ps.pin[g] = reinterpret_cast<const int32_t*>(arr(g ? kImgPin1 : kImgPin0));
    ps.rec[g] = g ? pp.rec1 : pp.rec0;
    ps.val[g] = reinterpret_cast<double*>(ws + (g ? L.val1 : L.val0));
  }
  ps.lnp2 = reinterpret_cast<double*>(ws + L.lnp);
  ps.bad = p1.clear_flags;
  ps.status = reinterpret_cast<int32_t*>(ws + L.status);
  ps.loss = loss_out;
  if (launch_arc_sweep(plan->state_chunks, plan->slots_per_state, ps, stream) != hipSuccess) return RNNT_ERR_HIP;
  if (mark(3) != hipSuccess) return RNNT_ERR_HIP;

  ArcRowParams pr{};
  pr.T_max = shape.T_max;
  pr.U_max = shape.U_max;
  pr.blank = plan->blank;
  pr.n_rows = static_cast<int32_t>(n_rows);
  pr.n_arcs = plan->num_slots[0];
  pr.n_row_arcs = plan->num_row_arcs;
  pr.n_states = plan->num_states;
  pr.logit_lens = logit_lens;
  pr.label_lens = label_lens;
  pr.utt = ps.utt;
  pr.arcs = pp.arcs;
  pr.row_seg = reinterpret_cast<const int32_t*>(arr(kImgRowSeg));
  pr.row_arc = reinterpret_cast<const int32_t*>(arr(kImgRowArc));
  pr.rec0 = pp.rec0;
  pr.val0 = ps.val[0];
  pr.val1 = ps.val[1];
  pr.lnp2 = ps.lnp2;
  pr.status = ps.status;
  pr.lse2_rows = p1.lse2_rows;
  pr.rowinfo = reinterpret_cast<RowInfo*>(ws + L.rowinfo);
  pr.occ = reinterpret_cast<int2*>(ws + L.occ);
  if (grad_out && launch_arc_posteriors(pr, n_rows, stream) != hipSuccess) return RNNT_ERR_HIP;
  if (mark(4) != hipSuccess) return RNNT_ERR_HIP;

  if (grad_out) {
    GradParams p3{};
    p3.logits = logits;
    p3.grad = grad_out;
    p3.rowinfo = pr.rowinfo;
    p3.n_elem = n_rows * shape.V;
    p3.n_rows = n_rows;
    p3.V = shape.V;
    p3.blank = plan->blank;
    if (launch_grad(shape.dtype, shape.grad_dtype, p3, stream) != hipSuccess) return RNNT_ERR_HIP;
    ArcExtraParams px{};
    px.rows = pr;
    px.logits = logits;
    px.grad = grad_out;
    px.xrows = reinterpret_cast<const int32_t*>(arr(kImgXrows));
    px.V = shape.V;
    if (launch_arc_extra_rows(shape.dtype, shape.grad_dtype, px, plan->num_extra_rows, stream) != hipSuccess)
      return RNNT_ERR_HIP;
  }
  if (mark(5) != hipSuccess) return RNNT_ERR_HIP;
  return RNNT_OK;
}

rnnt_status_t rnnt_arc_loss(const void* logits, rnnt_shape_t shape, const int32_t* logit_lens,
                            const int32_t* label_lens, const rnnt_arc_plan_t* plan, const void* plan_image,
                            float* loss_out, void* grad_out, void* workspace, size_t workspace_bytes,
                            hipStream_t stream) {
  return rnnt_arc_loss_timed(logits, shape, logit_lens, label_lens, plan, plan_image, loss_out, grad_out, workspace,
                             workspace_bytes, stream, nullptr);
}

rnnt_status_t rnnt_log_softmax_gather(const void* logits, rnnt_shape_t shape, const int32_t* labels,
                                      const int32_t* logit_lens, const int32_t* label_lens,
                                      int32_t blank, double* lse_out, double* lp_blank_out,
                                      double* lp_label_out, hipStream_t stream) {
  rnnt_status_t st = check_shape(shape);
  if (st != RNNT_OK) return st;
  if (!logits || !logit_lens || !label_lens || !lp_blank_out || !lp_label_out || (!labels && shape.U_max > 0))
    return RNNT_ERR_NULL_PTR;
  if (blank < 0 || blank >= shape.V) return RNNT_ERR_BAD_BLANK;
  if (!aligned16(logits)) return RNNT_ERR_ALIGNMENT;
  const int64_t U1 = shape.U_max + 1;
  PopulateParams p1{};
  p1.logits = logits;
  p1.B = shape.B;
  p1.T_max = shape.T_max;
  p1.U_max = shape.U_max;
  p1.V = shape.V;
  p1.blank = blank;
  p1.labels = labels;
  p1.logit_lens = logit_lens;
  p1.label_lens = label_lens;
  p1.n_elem = static_cast<int64_t>(shape.B) * shape.T_max * U1 * shape.V;
  p1.lse_out = lse_out;
  p1.lp_blank_out = lp_blank_out;
  p1.lp_label_out = lp_label_out;
  return launch_populate_dense(shape.dtype, p1, stream) == hipSuccess ? RNNT_OK : RNNT_ERR_HIP;
}

rnnt_status_t rnnt_lattice_scores(const double* lp_blank, const double* lp_label, rnnt_shape_t shape,
                                  const int32_t* logit_lens, const int32_t* label_lens,
                                  rnnt_variant_t variant, double* alpha_out, double* beta_out,
                                  double* loss_out, double* loss_bwd_out, double* occ_blank_out,
                                  double* occ_label_out, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
  rnnt_shape_t s = shape;
  s.dtype = RNNT_DTYPE_F32;
  s.grad_dtype = RNNT_DTYPE_F32;
  rnnt_status_t st = check_shape(s);
  if (st != RNNT_OK) return st;
  if (!lp_blank || !lp_label || !logit_lens || !label_lens) return RNNT_ERR_NULL_PTR;
  if (!variant_known(variant)) return RNNT_ERR_BAD_VARIANT;
  if (!scores_fit(s)) return RNNT_ERR_UNSUPPORTED;
  const Layout L = make_layout(s, false);
  OwnedWorkspace owned;
  char* ws = nullptr;
  st = take_workspace(workspace, workspace_bytes, L.total, stream, owned, &ws);
  if (st != RNNT_OK) return st;

  LatticeParams p2{};
  p2.B = s.B;
  p2.T_max = s.T_max;
  p2.U_max = s.U_max;
  p2.V = s.V;
  p2.blank = 0;
  p2.labels = nullptr;
  p2.logit_lens = logit_lens;
  p2.label_lens = label_lens;
  p2.lp_blank = lp_blank;
  p2.lp_label = lp_label;
  p2.alpha = reinterpret_cast<double*>(ws + L.alpha);
  p2.beta = reinterpret_cast<double*>(ws + L.beta);
  p2.u_pad = 64 * units_per_lane(shape.U_max + 1);
  p2.lnp2_fwd = reinterpret_cast<double*>(ws + L.lnp);
  p2.lnp2_bwd = p2.lnp2_fwd + s.B;
  p2.status = reinterpret_cast<int32_t*>(ws + L.status);
  p2.loss_f32 = nullptr;
  if (launch_lattice_dense(variant, p2, stream) != hipSuccess) return RNNT_ERR_HIP;

  PostParams pb{};
  pb.B = s.B;
  pb.T_max = s.T_max;
  pb.U_max = s.U_max;
  pb.labels = nullptr;
  pb.logit_lens = logit_lens;
  pb.label_lens = label_lens;
  pb.status = p2.status;
  pb.lp_blank = lp_blank;
  pb.lp_label = lp_label;
  pb.alpha = p2.alpha;
  pb.beta = p2.beta;
  pb.u_pad = p2.u_pad;
  pb.lnp2_fwd = p2.lnp2_fwd;
  pb.lnp2_bwd = p2.lnp2_bwd;
  pb.n_rows = static_cast<int64_t>(s.B) * s.T_max * (s.U_max + 1);
  pb.alpha_out = alpha_out;
  pb.beta_out = beta_out;
  pb.occ_blank_out = occ_blank_out;
  pb.occ_label_out = occ_label_out;
  pb.loss_out = loss_out;
  pb.loss_bwd_out = loss_bwd_out;
  return launch_posteriors_dense(pb, stream) == hipSuccess ? RNNT_OK : RNNT_ERR_HIP;
}

}  // extern "C"
