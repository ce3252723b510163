// C-ABI entry points of libfcngrad: host-side validation, the lowering of
// each convolution pass onto the implicit-GEMM kernels, and the host-only
// helpers. Every check runs before the first HIP call, so an invalid call
// returns without touching the device.
#include <string.h>

#include <algorithm>
#include <cmath>
#include <mutex>
#include <unordered_map>

#include "internal.h"

using namespace fg;

namespace {

constexpr int64_t kMaxElems = (int64_t)1 << 31;

bool pos(int32_t v) { return v > 0; }

int64_t elems4(int64_t a, int64_t b, int64_t c, int64_t d) {
  return a * b * c * d;
}

// Forward output size; <= 0 when the kernel does not fit.
int32_t fwd_out(int32_t in, int32_t pad, int32_t ker, int32_t str) {
  int64_t t = (int64_t)in + 2 * (int64_t)pad - ker;
  if (t < 0) return 0;
  return (int32_t)(t / str + 1);
}

int32_t convt_out(int32_t in, int32_t pad, int32_t ker, int32_t str) {
  int64_t o = ((int64_t)in - 1) * str - 2 * (int64_t)pad + ker;
  return o > 0 && o < kMaxElems ? (int32_t)o : 0;
}

fg_status check_desc(const fg_conv_desc *d) {
  if (!d) return FG_EINVAL;
  if (!pos(d->n) || !pos(d->h) || !pos(d->w) || !pos(d->c) || !pos(d->k) ||
      !pos(d->r) || !pos(d->s) || !pos(d->stride_h) || !pos(d->stride_w) ||
      d->pad_h < 0 || d->pad_w < 0 || d->x_ld < 0 || d->y_ld < 0)
    return FG_EINVAL;
  return FG_OK;
}

// K == 1 is served by the bandwidth kernels of the 1x1 head only.
bool is_head(const fg_conv_desc *d) {
  return d->k == 1 && d->r == 1 && d->s == 1 && d->stride_h == 1 &&
         d->stride_w == 1 && d->pad_h == 0 && d->pad_w == 0;
}

fg_status check_conv_support(const fg_conv_desc *d) {
  if (d->c % 8 != 0) return FG_EUNSUPPORTED;
  if (d->k == 1) return is_head(d) && d->c <= 2048 ? FG_OK : FG_EUNSUPPORTED;
  if (d->k % 8 != 0) return FG_EUNSUPPORTED;
  if (d->r * d->s > 16) return FG_EUNSUPPORTED;
  return FG_OK;
}

// Byte ranges [a, a+na) and [b, b+nb) overlap.
bool overlap(const void *a, size_t na, const void *b, size_t nb) {
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

// A ReLU-gradient gate has the output's layout and is read at each output
// element by the thread that then writes that element: it may be the output
// itself, but no other overlap (another workgroup could overwrite a gate
// value before it is read).
bool gate_ok(const void *gate, const void *out, size_t span) {
  return gate == nullptr || gate == out || !overlap(gate, span, out, span);
}

bool sizes_ok(int64_t a, int64_t b, int64_t c) {
  return a < kMaxElems && b < kMaxElems && c < kMaxElems;
}

fg_status launch_status(hipError_t e) {
  return e == hipSuccess ? FG_OK : FG_ELAUNCH;
}

// Pixel stride (elements) of a tensor with ch channels: ld, 0 meaning dense.
int64_t ld_or(int32_t ld, int32_t ch) { return ld ? ld : ch; }

// Inputs are read dense.
bool dense_ld(int32_t ld, int32_t ch) { return ld == 0 || ld == ch; }

// An output written at pixel stride ld: dense, or ld >= ch, a multiple of 8
// elements, a 16-byte aligned pointer and npix * ld below 2^31.
fg_status out_ld_ok(int32_t ld, int32_t ch, int64_t npix, const void *p) {
  if (dense_ld(ld, ch)) return FG_OK;
  if (ld < ch) return FG_EINVAL;
  if (ld % 8 != 0 || ((uintptr_t)p & 15) != 0) return FG_EUNSUPPORTED;
  if (npix * (int64_t)ld >= kMaxElems) return FG_EUNSUPPORTED;
  return FG_OK;
}

// Bytes from the first to the last element of npix pixels at stride ld.
size_t span_bytes(int64_t npix, int64_t ld, int64_t ch) {
  return (size_t)((npix - 1) * ld + ch) * 2;
}

// Two channel slices at one pixel stride ld: ch1 channels from a, ch2 from
// b. Their elements are disjoint, whatever their pixel ranges, when b's
// first channel lies at least ch1 channels past a's and its last one before
// a's next pixel (b - a taken modulo the pixel stride).
bool slices_disjoint(const void *a, int64_t ch1, const void *b, int64_t ch2,
                     int64_t ld) {
  const int64_t db = (int64_t)((uintptr_t)b - (uintptr_t)a);
  if (db % 2 != 0) return false;
  const int64_t r = ((db / 2) % ld + ld) % ld;
  return ch1 <= r && r + ch2 <= ld;
}

// Overlap of an input slice (x, npx pixels at stride ldx, cx channels) with
// an output slice (y, npy at ldy, cy): interleaved slices of one buffer
// (a dense block's layer reading the channels before the ones it writes)
// do not overlap.
bool slices_overlap(const void *x, int64_t npx, int64_t ldx, int64_t cx,
                    const void *y, int64_t npy, int64_t ldy, int64_t cy) {
  if (ldx == ldy && slices_disjoint(x, cx, y, cy, ldx)) return false;
  return overlap(x, span_bytes(npx, ldx, cx), y, span_bytes(npy, ldy, cy));
}

bool epi_ok(int epi) {
  return epi == FG_EPI_NONE || epi == FG_EPI_RELU || epi == FG_EPI_GATE ||
         epi == FG_EPI_ACC;
}

// Phase description for an input-gradient style convolution (scatter form
// evaluated per output phase). Dimension of size `out` with stride `str`,
// padding `pad`, kernel `ker`, input (gathered) size `in`: for output
// positions o = a*str + ph, the taps are r = r0, r0+str, ... with
// (ph + pad - r) divisible by str, reading input row a + (ph + pad - r)/str.
struct Dim1 {
  int32_t m, r0, n, d0;
};

Dim1 phase_dim(int32_t out, int32_t str, int32_t pad, int32_t ker,
               int32_t ph) {
  Dim1 d{0, 0, 0, 0};
  d.m = ph < out ? (out - ph + str - 1) / str : 0;
  int32_t r0 = ((ph + pad) % str + str) % str;
  d.r0 = r0;
  d.n = r0 < ker ? (ker - r0 + str - 1) / str : 0;
  d.d0 = (ph + pad - r0) / str;  // exact: ph + pad - r0 is a multiple of str
  return d;
}

// Fill the phases of an input-gradient style lowering. Returns the count.
int make_phases(DataConvArgs &a, int32_t ho, int32_t wo, int32_t sh,
                int32_t sw, int32_t pad_h, int32_t pad_w, int32_t r,
                int32_t s) {
  int np = 0;
  for (int ph = 0; ph < sh; ++ph)
    for (int pw = 0; pw < sw; ++pw) {
      Dim1 dh = phase_dim(ho, sh, pad_h, r, ph);
      Dim1 dw = phase_dim(wo, sw, pad_w, s, pw);
      Phase &P = a.ph[np++];
      P.mh = dh.m;
      P.mw = dw.m;
      P.ooh = ph;
      P.oow = pw;
      P.nr = dh.n;
      P.ns = dw.n;
      P.dh0 = dh.d0;
      P.dw0 = dw.d0;
      P.dstep = -1;
      P.r0 = dh.r0;
      P.s0 = dw.r0;
      P.rstep = sh;  // equal strides only (checked by the callers)
    }
  return np;
}

// Argument builders shared by the launch, workspace and kernel-name paths.
DataConvArgs fwd_args(const fg_conv_desc *d, int32_t P, int32_t Q) {
  DataConvArgs a;
  memset(&a, 0, sizeof(a));
  a.n = d->n; a.hi = d->h; a.wi = d->w; a.cr = d->c;
  a.ldi = (int32_t)ld_or(d->x_ld, d->c);
  a.ho = P; a.wo = Q; a.co = d->k;
  a.ldo = (int32_t)ld_or(d->y_ld, d->k);
  a.istr = d->stride_h;
  a.ostr = 1;
  a.s = d->s;
  a.ldw = d->r * d->s * d->c;
  a.wbytes = (int32_t)std::min<int64_t>(elems4(d->k, d->r, d->s, d->c) * 2,
                                        0x7FFFFFFF);
  a.nphase = 1;
  a.nsplit = 1;
  Phase &ph = a.ph[0];
  ph.mh = P; ph.mw = Q; ph.ooh = 0; ph.oow = 0;
  ph.nr = d->r; ph.ns = d->s;
  ph.dh0 = -d->pad_h; ph.dw0 = -d->pad_w; ph.dstep = 1;
  ph.r0 = 0; ph.s0 = 0; ph.rstep = 1;
  return a;
}

DataConvArgs bwd_data_args(const fg_conv_desc *d, int32_t P, int32_t Q) {
  DataConvArgs a;
  memset(&a, 0, sizeof(a));
  a.n = d->n; a.hi = P; a.wi = Q; a.cr = d->k;
  a.ldi = d->k;
  a.ho = d->h; a.wo = d->w; a.co = d->c;
  a.ldo = (int32_t)ld_or(d->x_ld, d->c);
  a.istr = 1;
  a.ostr = d->stride_h;
  a.s = d->s;
  a.w_red = d->r * d->s * d->c;  // W[k][r][s][c]: reduction index k
  a.w_tap = d->c;
  a.wbytes = (int32_t)std::min<int64_t>(elems4(d->k, d->r, d->s, d->c) * 2,
                                        0x7FFFFFFF);
  a.nsplit = 1;
  a.nphase = make_phases(a, d->h, d->w, d->stride_h, d->stride_w, d->pad_h,
                         d->pad_w, d->r, d->s);
  return a;
}

DataConvArgs convt_args(const fg_conv_desc *d, int32_t HO, int32_t WO) {
  DataConvArgs a;
  memset(&a, 0, sizeof(a));
  a.n = d->n; a.hi = d->h; a.wi = d->w; a.cr = d->c;
  a.ldi = d->c;
  a.ho = HO; a.wo = WO; a.co = d->k;
  a.ldo = (int32_t)ld_or(d->y_ld, d->k);
  a.istr = 1;
  a.ostr = d->stride_h;
  a.s = d->s;
  a.w_red = d->r * d->s * d->k;  // Wt[c][r][s][k]: reduction index c
  a.w_tap = d->k;
  a.wbytes = (int32_t)std::min<int64_t>(elems4(d->c, d->r, d->s, d->k) * 2,
                                        0x7FFFFFFF);
  a.nsplit = 1;
  a.nphase = make_phases(a, HO, WO, d->stride_h, d->stride_w, d->pad_h,
                         d->pad_w, d->r, d->s);
  return a;
}

bool convt_supported(const fg_conv_desc *d) {
  return d->c % 8 == 0 && d->k % 8 == 0 && d->r == 4 && d->s == 4 &&
         d->stride_h == 2 && d->stride_w == 2 && d->pad_h == 1 &&
         d->pad_w == 1;
}

bool bwd_data_supported(const fg_conv_desc *d) {
  return check_conv_support(d) == FG_OK && d->stride_h == d->stride_w &&
         d->stride_h <= 2;
}

bool fwd_supported(const fg_conv_desc *d) {
  return check_conv_support(d) == FG_OK && d->stride_h == d->stride_w;
}

// Workspace of a data convolution pass (0 when it does not split).
size_t data_ws(const fg_conv_desc *d, int op) {
  int32_t p, q;
  if (op == FG_OP_CONVT) {
    if (!convt_supported(d) || fg_conv_out_dims(d, 1, &p, &q) != FG_OK) return 0;
    return plan_data_conv(convt_args(d, p, q)).ws_bytes;
  }
  if (fg_conv_out_dims(d, 0, &p, &q) != FG_OK || d->k == 1) return 0;
  if (op == FG_OP_FWD)
    return fwd_supported(d) ? plan_data_conv(fwd_args(d, p, q)).ws_bytes : 0;
  return bwd_data_supported(d) ? plan_data_conv(bwd_data_args(d, p, q)).ws_bytes
                               : 0;
}

// Workspace present and large enough, and not overlapping the tensors
// (byte ranges (p_i, n_i)).
fg_status check_ws_need(size_t need, void *ws, size_t ws_bytes,
                        const void *p0, size_t n0, const void *p1, size_t n1,
                        const void *p2, size_t n2, const void *p3, size_t n3) {
  if (need == 0) return FG_OK;
  if (!ws || ws_bytes < need) return FG_EWORKSPACE;
  if (overlap(ws, need, p0, n0) || overlap(ws, need, p1, n1) ||
      (p2 && overlap(ws, need, p2, n2)) || (p3 && overlap(ws, need, p3, n3)))
    return FG_EINVAL;
  return FG_OK;
}

fg_status check_ws(const fg_conv_desc *d, int op, void *ws, size_t ws_bytes,
                   const void *p0, size_t n0, const void *p1, size_t n1,
                   const void *p2, size_t n2, const void *p3, size_t n3) {
  return check_ws_need(fg_conv_workspace_bytes(d, op), ws, ws_bytes, p0, n0, p1,
                       n1, p2, n2, p3, n3);
}

// ---- the no-allocation kernel gradient's scratch ---------------------------
// fp32 split partials of conv2d_bwd_weight_noalloc. Each GPU the library runs
// on holds its own copy until the process ends. In host code the array's name
// is only a host-side stand-in: its device address on the current device is
// looked up once per device with hipGetSymbolAddress, and only that address is
// handed to kernels.
static __device__ __align__(256) unsigned char scratch[FG_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];  // device address of `scratch`, per device

// Device address of `scratch` on the current device (looked up on the first
// call on each device, with that device current).
fg_status scratch_for_current_device(void **out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices)
    return FG_ELAUNCH;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p)
      return FG_ELAUNCH;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return FG_OK;
}

}  // namespace

// ---------------------------------------------------------------------------
extern "C" {

const char *fg_status_string(fg_status s) {
  switch (s) {
    case FG_OK: return "FG_OK";
    case FG_EINVAL: return "FG_EINVAL: invalid argument";
    case FG_EUNSUPPORTED: return "FG_EUNSUPPORTED: shape not implemented";
    case FG_EWORKSPACE: return "FG_EWORKSPACE: workspace too small";
    case FG_ELAUNCH: return "FG_ELAUNCH: kernel launch failed";
  }
  return "unknown fg_status";
}

fg_status fg_conv_out_dims(const fg_conv_desc *d, int transpose, int32_t *p,
                           int32_t *q) {
  if (check_desc(d) != FG_OK || !p || !q || (transpose != 0 && transpose != 1))
    return FG_EINVAL;
  int32_t pp, qq;
  if (transpose) {
    pp = convt_out(d->h, d->pad_h, d->r, d->stride_h);
    qq = convt_out(d->w, d->pad_w, d->s, d->stride_w);
  } else {
    pp = fwd_out(d->h, d->pad_h, d->r, d->stride_h);
    qq = fwd_out(d->w, d->pad_w, d->s, d->stride_w);
  }
  if (pp <= 0 || qq <= 0) return FG_EINVAL;
  *p = pp;
  *q = qq;
  return FG_OK;
}

size_t fg_conv_workspace_bytes(const fg_conv_desc *d, int op) {
  if (check_desc(d) != FG_OK) return 0;
  if (op == FG_OP_BWD_WEIGHT) {
    int32_t p, q;
    if (fg_conv_out_dims(d, 0, &p, &q) != FG_OK) return 0;
    if (check_conv_support(d) != FG_OK) return 0;
    if (is_head(d)) return head_wgrad_ws_bytes(*d);
    return plan_wgrad(*d, p, q).ws_bytes;
  }
  if (op == FG_OP_FWD || op == FG_OP_BWD_DATA || op == FG_OP_CONVT)
    return data_ws(d, op);
  return 0;
}

const char *fg_conv_kernel_name(const fg_conv_desc *d, int op) {
  if (check_desc(d) != FG_OK) return "";
  int32_t p, q;
  switch (op) {
    case FG_OP_FWD:
      if (!fwd_supported(d) || fg_conv_out_dims(d, 0, &p, &q) != FG_OK) return "";
      return d->k == 1 ? "head_fwd_kernel"
                       : data_conv_kernel_name(fwd_args(d, p, q), true);
    case FG_OP_BWD_DATA:
      if (!bwd_data_supported(d) || fg_conv_out_dims(d, 0, &p, &q) != FG_OK)
        return "";
      return d->k == 1 ? "head_bwd_data_kernel"
                       : data_conv_kernel_name(bwd_data_args(d, p, q), false);
    case FG_OP_BWD_WEIGHT:
      if (check_conv_support(d) != FG_OK) return "";
      return d->k == 1 ? "head_wgrad_kernel" : wgrad_kernel_name(*d);
    case FG_OP_CONVT:
      if (!convt_supported(d) || fg_conv_out_dims(d, 1, &p, &q) != FG_OK) return "";
      return data_conv_kernel_name(convt_args(d, p, q), false);
  }
  return "";
}

fg_status conv2d_fwd(const fg_conv_desc *d, const uint16_t *x,
                     const uint16_t *w_krsc, uint16_t *y, fg_epilogue epi,
                     const uint16_t *gate, void *ws, size_t ws_bytes,
                     hipStream_t stream) {
  fg_status st = check_desc(d);
  if (st != FG_OK) return st;
  if (!x || !w_krsc || !y) return FG_EINVAL;
  if (!epi_ok(epi)) return FG_EINVAL;
  if (epi == FG_EPI_GATE && !gate) return FG_EINVAL;
  int32_t P, Q;
  if (fg_conv_out_dims(d, 0, &P, &Q) != FG_OK) return FG_EINVAL;
  const int64_t nx = elems4(d->n, d->h, d->w, d->c);
  const int64_t nw = elems4(d->k, d->r, d->s, d->c);
  const int64_t ny = elems4(d->n, P, Q, d->k);
  if (!sizes_ok(nx, nw, ny)) return FG_EUNSUPPORTED;
  const int64_t npx = (int64_t)d->n * d->h * d->w;
  const int64_t npy = (int64_t)d->n * P * Q;
  // the input may be a channel prefix of a wider buffer, like the output
  if ((st = out_ld_ok(d->x_ld, d->c, npx, x)) != FG_OK) return st;
  if ((st = out_ld_ok(d->y_ld, d->k, npy, y)) != FG_OK) return st;
  const int64_t ldx = ld_or(d->x_ld, d->c), ldy = ld_or(d->y_ld, d->k);
  const size_t sx = span_bytes(npx, ldx, d->c);
  const size_t sy = span_bytes(npy, ldy, d->k);
  if (slices_overlap(x, npx, ldx, d->c, y, npy, ldy, d->k) ||
      overlap(y, sy, w_krsc, nw * 2))
    return FG_EINVAL;
  if (epi == FG_EPI_GATE && !gate_ok(gate, y, sy)) return FG_EINVAL;
  if ((st = check_conv_support(d)) != FG_OK) return st;
  // one input step per output position for both image axes
  if (d->stride_h != d->stride_w) return FG_EUNSUPPORTED;

  if (d->k == 1) {
    if (!dense_ld(d->x_ld, d->c) || !dense_ld(d->y_ld, d->k) || epi == FG_EPI_ACC)
      return FG_EUNSUPPORTED;
    return launch_status(launch_head_fwd(x, w_krsc, y, (int64_t)d->n * P * Q,
                                         d->c, epi, gate, stream));
  }
  if ((st = check_ws(d, FG_OP_FWD, ws, ws_bytes, x, sx, w_krsc, nw * 2, y,
                     sy, gate, sy)) != FG_OK)
    return st;
  DataConvArgs a = fwd_args(d, P, Q);
  a.act = x;
  a.wgt = w_krsc;
  a.out = y;
  a.gate = gate;
  a.epi = epi;
  a.part = (float *)ws;
  return launch_status(launch_data_conv(a, true, stream));
}

fg_status conv2d_bwd_data(const fg_conv_desc *d, const uint16_t *dy,
                          const uint16_t *w_krsc, uint16_t *dx,
                          fg_epilogue epi, const uint16_t *gate, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
  fg_status st = check_desc(d);
  if (st != FG_OK) return st;
  if (!dy || !w_krsc || !dx) return FG_EINVAL;
  if (!epi_ok(epi)) return FG_EINVAL;
  if (epi == FG_EPI_GATE && !gate) return FG_EINVAL;
  int32_t P, Q;
  if (fg_conv_out_dims(d, 0, &P, &Q) != FG_OK) return FG_EINVAL;
  const int64_t nx = elems4(d->n, d->h, d->w, d->c);
  const int64_t nw = elems4(d->k, d->r, d->s, d->c);
  const int64_t ny = elems4(d->n, P, Q, d->k);
  if (!sizes_ok(nx, nw, ny)) return FG_EUNSUPPORTED;
  if (!dense_ld(d->y_ld, d->k)) return FG_EUNSUPPORTED;
  const int64_t npx = (int64_t)d->n * d->h * d->w;
  if ((st = out_ld_ok(d->x_ld, d->c, npx, dx)) != FG_OK) return st;
  const size_t sx = span_bytes(npx, ld_or(d->x_ld, d->c), d->c);
  if (overlap(dx, sx, dy, ny * 2) || overlap(dx, sx, w_krsc, nw * 2))
    return FG_EINVAL;
  if (epi == FG_EPI_GATE && !gate_ok(gate, dx, sx)) return FG_EINVAL;
  if ((st = check_conv_support(d)) != FG_OK) return st;
  if (d->stride_h != d->stride_w || d->stride_h > 2) return FG_EUNSUPPORTED;

  if (d->k == 1) {
    if (!dense_ld(d->x_ld, d->c) || epi == FG_EPI_ACC) return FG_EUNSUPPORTED;
    return launch_status(launch_head_bwd_data(
        dy, w_krsc, dx, (int64_t)d->n * d->h * d->w, d->c, epi, gate, stream));
  }
  if ((st = check_ws(d, FG_OP_BWD_DATA, ws, ws_bytes, dy, ny * 2, w_krsc, nw * 2,
                     dx, sx, gate, sx)) != FG_OK)
    return st;
  DataConvArgs a = bwd_data_args(d, P, Q);
  a.act = dy;
  a.wgt = w_krsc;
  a.out = dx;
  a.gate = gate;
  a.epi = epi;
  a.part = (float *)ws;
  return launch_status(launch_data_conv(a, false, stream));
}

fg_status conv_transpose2d_fwd(const fg_conv_desc *d, const uint16_t *x,
                               const uint16_t *w_crsk, uint16_t *y,
                               fg_epilogue epi, const uint16_t *gate,
                               void *ws, size_t ws_bytes, hipStream_t stream) {
  fg_status st = check_desc(d);
  if (st != FG_OK) return st;
  if (!x || !w_crsk || !y) return FG_EINVAL;
  if (!epi_ok(epi)) return FG_EINVAL;
  if (epi == FG_EPI_GATE && !gate) return FG_EINVAL;
  int32_t HO, WO;
  if (fg_conv_out_dims(d, 1, &HO, &WO) != FG_OK) return FG_EINVAL;
  const int64_t nx = elems4(d->n, d->h, d->w, d->c);
  const int64_t nw = elems4(d->c, d->r, d->s, d->k);
  const int64_t ny = elems4(d->n, HO, WO, d->k);
  if (!sizes_ok(nx, nw, ny)) return FG_EUNSUPPORTED;
  if (!dense_ld(d->x_ld, d->c)) return FG_EUNSUPPORTED;
  const int64_t npy = (int64_t)d->n * HO * WO;
  if ((st = out_ld_ok(d->y_ld, d->k, npy, y)) != FG_OK) return st;
  const size_t sy = span_bytes(npy, ld_or(d->y_ld, d->k), d->k);
  if (overlap(y, sy, x, nx * 2) || overlap(y, sy, w_crsk, nw * 2))
    return FG_EINVAL;
  if (epi == FG_EPI_GATE && !gate_ok(gate, y, sy)) return FG_EINVAL;
  if (!convt_supported(d)) return FG_EUNSUPPORTED;
  if ((st = check_ws(d, FG_OP_CONVT, ws, ws_bytes, x, nx * 2, w_crsk, nw * 2, y,
                     sy, gate, sy)) != FG_OK)
    return st;
  DataConvArgs a = convt_args(d, HO, WO);
  a.act = x;
  a.wgt = w_crsk;
  a.out = y;
  a.gate = gate;
  a.epi = epi;
  a.part = (float *)ws;
  return launch_status(launch_data_conv(a, false, stream));
}

// noalloc: the split partials go to the library's static scratch (ws and
// ws_bytes are ignored) and the plan keeps them within its size.
static fg_status bwd_weight(const fg_conv_desc *d, const uint16_t *x,
                            const uint16_t *dy, uint16_t *dw_krsc,
                            int32_t *found_nonfinite, void *ws, size_t ws_bytes,
                            hipStream_t stream, bool noalloc = false) {
  fg_status st = check_desc(d);
  if (st != FG_OK) return st;
  if (!x || !dy || !dw_krsc) return FG_EINVAL;
  if (!dense_ld(d->y_ld, d->k)) return FG_EUNSUPPORTED;
  int32_t P, Q;
  if (fg_conv_out_dims(d, 0, &P, &Q) != FG_OK) return FG_EINVAL;
  const int64_t nx = elems4(d->n, d->h, d->w, d->c);
  // x may be a channel prefix of a wider buffer; sx is its span
  const int64_t npx = (int64_t)d->n * d->h * d->w;
  if (out_ld_ok(d->x_ld, d->c, npx, x) != FG_OK) return out_ld_ok(d->x_ld, d->c, npx, x);
  if (d->k == 1 && !dense_ld(d->x_ld, d->c)) return FG_EUNSUPPORTED;
  const size_t sx = span_bytes(npx, ld_or(d->x_ld, d->c), d->c);
  const int64_t nw = elems4(d->k, d->r, d->s, d->c);
  const int64_t ny = elems4(d->n, P, Q, d->k);
  if (!sizes_ok(nx, nw, ny)) return FG_EUNSUPPORTED;
  if (overlap(dw_krsc, nw * 2, x, sx) ||
      overlap(dw_krsc, nw * 2, dy, ny * 2))
    return FG_EINVAL;
  if (found_nonfinite &&
      (overlap(found_nonfinite, 4, dw_krsc, nw * 2) ||
       overlap(found_nonfinite, 4, x, sx) ||
       overlap(found_nonfinite, 4, dy, ny * 2) ||
       overlap(found_nonfinite, 4, ws, ws_bytes)))
    return FG_EINVAL;
  if ((st = check_conv_support(d)) != FG_OK) return st;
  const size_t plan_cap = noalloc ? (size_t)FG_NOALLOC_SCRATCH_BYTES : SIZE_MAX;
  const size_t need = d->k == 1 ? head_wgrad_ws_bytes(*d)
                                : plan_wgrad(*d, P, Q, plan_cap).ws_bytes;
  if (noalloc) {
    // the library's scratch cannot overlap the caller's buffers
    if (need > (size_t)FG_NOALLOC_SCRATCH_BYTES) return FG_EWORKSPACE;
    ws = nullptr;
    ws_bytes = 0;
    if (need && (st = scratch_for_current_device(&ws)) != FG_OK) return st;
    ws_bytes = FG_NOALLOC_SCRATCH_BYTES;
  } else if ((st = check_ws_need(need, ws, ws_bytes, x, sx, dy, ny * 2, dw_krsc,
                                 nw * 2, nullptr, 0)) != FG_OK) {
    return st;
  }

  if (d->k == 1)
    return launch_status(launch_head_wgrad(x, dy, dw_krsc,
                                           (int64_t)d->n * d->h * d->w, d->c,
                                           (float *)ws, found_nonfinite, stream));
  WgradPlan pl = plan_wgrad(*d, P, Q, plan_cap);
  WgradArgs a;
  memset(&a, 0, sizeof(a));
  a.x = x;
  a.dy = dy;
  a.dw = dw_krsc;
  a.part = (float *)ws;
  a.n = d->n; a.h = d->h; a.w = d->w; a.c = d->c; a.k = d->k;
  a.ldx = (int32_t)ld_or(d->x_ld, d->c);
  a.r = d->r; a.s = d->s; a.p = P; a.q = Q;
  a.sh = d->stride_h; a.sw = d->stride_w; a.ph = d->pad_h; a.pw = d->pad_w;
  a.mtot = d->n * P * Q;
  a.mchunk = pl.mchunk;
  a.nsplit = pl.nsplit;
  a.flag = found_nonfinite;
  return launch_status(launch_wgrad(a, pl.big, stream));
}

fg_status conv2d_bwd_weight(const fg_conv_desc *d, const uint16_t *x,
                            const uint16_t *dy, uint16_t *dw_krsc, void *ws,
                            size_t ws_bytes, hipStream_t stream) {
  return bwd_weight(d, x, dy, dw_krsc, nullptr, ws, ws_bytes, stream);
}

fg_status conv2d_bwd_weight_checked(const fg_conv_desc *d, const uint16_t *x,
                                    const uint16_t *dy, uint16_t *dw_krsc,
                                    int32_t *found_nonfinite, void *ws,
                                    size_t ws_bytes, hipStream_t stream) {
  if (!found_nonfinite) return FG_EINVAL;
  return bwd_weight(d, x, dy, dw_krsc, found_nonfinite, ws, ws_bytes, stream);
}

fg_status conv2d_bwd_weight_noalloc(const fg_conv_desc *d, const uint16_t *x,
                                    const uint16_t *dy, uint16_t *dw_krsc,
                                    hipStream_t stream) {
  return bwd_weight(d, x, dy, dw_krsc, nullptr, nullptr, 0, stream, true);
}

// ---------------------------------------------------------------------------
// Segments must lie inside the group and not overlap there; with
// distinct_ptrs (unpack destinations) their device ranges must not overlap
// either.
static fg_status check_segments(const fg_segment *segs, int32_t nseg,
                                uint64_t group_numel, size_t esz,
                                bool distinct_ptrs) {
  if (!segs || nseg < 1) return FG_EINVAL;
  if (nseg > FG_MAX_SEGMENTS) return FG_EUNSUPPORTED;
  if (group_numel >= (uint64_t)kMaxElems) return FG_EUNSUPPORTED;
  for (int i = 0; i < nseg; ++i) {
    const fg_segment &s = segs[i];
    if (!s.ptr && s.numel) return FG_EINVAL;
    if (s.offset > group_numel || s.numel > group_numel - s.offset)
      return FG_EINVAL;
    for (int j = 0; j < i; ++j) {
      const fg_segment &t = segs[j];
      if (s.numel && t.numel && s.offset < t.offset + t.numel &&
          t.offset < s.offset + s.numel)
        return FG_EINVAL;
      if (distinct_ptrs && s.numel && t.numel &&
          overlap((void *)s.ptr, s.numel * esz, (void *)t.ptr, t.numel * esz))
        return FG_EINVAL;
    }
  }
  return FG_OK;
}

fg_status grad_group_pack(const fg_segment *segs, int32_t nseg,
                          uint16_t *group, uint64_t group_numel,
                          hipStream_t stream) {
  if (!group || group_numel == 0) return FG_EINVAL;
  fg_status st = check_segments(segs, nseg, group_numel, 2, false);
  if (st != FG_OK) return st;
  for (int i = 0; i < nseg; ++i)
    if (overlap((void *)segs[i].ptr, segs[i].numel * 2, group, group_numel * 2))
      return FG_EINVAL;
  return launch_status(launch_pack(segs, nseg, group, group_numel, stream));
}

fg_status grad_group_unpack(const float *group_f32, uint64_t group_numel,
                            const fg_segment *segs, int32_t nseg,
                            hipStream_t stream) {
  if (!group_f32 || group_numel == 0) return FG_EINVAL;
  fg_status st = check_segments(segs, nseg, group_numel, 4, true);
  if (st != FG_OK) return st;
  for (int i = 0; i < nseg; ++i)
    if (overlap((void *)segs[i].ptr, segs[i].numel * 4, group_f32,
                group_numel * 4))
      return FG_EINVAL;
  return launch_status(launch_unpack(group_f32, segs, nseg, stream));
}

fg_status grad_flags_clear(int32_t *flags, int32_t n, hipStream_t stream) {
  if (!flags || n < 1) return FG_EINVAL;
  return launch_status(launch_flags_clear(flags, n, stream));
}

fg_status grad_unscale_check(const uint16_t *group, uint64_t numel,
                             float inv_scale, float *out_f32,
                             int32_t *found_nonfinite, hipStream_t stream) {
  if (!group || !out_f32 || !found_nonfinite || numel == 0) return FG_EINVAL;
  if (numel >= (uint64_t)kMaxElems) return FG_EUNSUPPORTED;
  if (overlap(group, numel * 2, out_f32, numel * 4) ||
      overlap(found_nonfinite, 4, out_f32, numel * 4) ||
      overlap(found_nonfinite, 4, group, numel * 2))
    return FG_EINVAL;
  return launch_status(launch_unscale(group, numel, inv_scale, out_f32,
                                      found_nonfinite, stream));
}

// ---------------------------------------------------------------------------
// gbytes: bytes per gradient element (4: fp32, 2: fp16)
static bool opt_tensors_ok(const fg_opt_tensor *t, int32_t n, size_t gbytes = 4) {
  if (!t || n < 1 || n > FG_MAX_SEGMENTS) return false;
  const uint64_t galign = gbytes == 4 ? 15 : 7;
  for (int i = 0; i < n; ++i) {
    const fg_opt_tensor &a = t[i];
    if (!a.w32 || !a.w16 || !a.m || !a.v || !a.g) return false;
    if (a.numel == 0 || a.numel >= 0x7FFFFFFFull) return false;
    if (((a.w32 | a.m | a.v) & 15) || (a.g & galign) || (a.w16 & 7)) return false;
  }
  // no two arrays of the call overlap
  const size_t bytes[5] = {4, 4, 4, gbytes, 2};
  for (int i = 0; i < n; ++i) {
    const uint64_t pi[5] = {t[i].w32, t[i].m, t[i].v, t[i].g, t[i].w16};
    for (int j = i; j < n; ++j) {
      const uint64_t pj[5] = {t[j].w32, t[j].m, t[j].v, t[j].g, t[j].w16};
      for (int a = 0; a < 5; ++a)
        for (int b = (i == j ? a + 1 : 0); b < 5; ++b)
          if (overlap((const void *)pi[a], t[i].numel * bytes[a], (const void *)pj[b],
                      t[j].numel * bytes[b]))
            return false;
    }
  }
  return true;
}

static bool opt_params_ok(const fg_opt_params *p) {
  return p && std::isfinite(p->lr) && p->lr >= 0.f && std::isfinite(p->beta1) &&
         p->beta1 >= 0.f && p->beta1 < 1.f && std::isfinite(p->beta2) &&
         p->beta2 >= 0.f && p->beta2 < 1.f && std::isfinite(p->eps) && p->eps >= 0.f &&
         std::isfinite(p->weight_decay) && p->weight_decay >= 0.f;
}

// Shared checks of the optimizer calls: the table, the gradient format, the
// step count and the workspace (size, alignment, no aliasing of any array).
static fg_status opt_call_ok(const fg_opt_tensor *t, int32_t n, const fg_opt_params *p,
                             int32_t grad_format, float inv_scale,
                             const int32_t *step_count, const void *ws,
                             size_t ws_bytes) {
  if (grad_format != FG_GRAD_F32 && grad_format != FG_GRAD_F16_SCALED) return FG_EINVAL;
  if (grad_format == FG_GRAD_F16_SCALED && !(std::isfinite(inv_scale) && inv_scale > 0.f))
    return FG_EINVAL;
  const size_t gb = grad_format == FG_GRAD_F32 ? 4 : 2;
  if (!opt_tensors_ok(t, n, gb) || !opt_params_ok(p) || !step_count) return FG_EINVAL;
  const size_t need = lars_adam_ws_bytes(t, n);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 15)) return FG_EWORKSPACE;
  const size_t bytes[5] = {4, 4, 4, gb, 2};
  for (int i = 0; i < n; ++i) {
    const uint64_t pa[5] = {t[i].w32, t[i].m, t[i].v, t[i].g, t[i].w16};
    for (int a = 0; a < 5; ++a) {
      if (overlap((const void *)pa[a], t[i].numel * bytes[a], step_count, 4) ||
          overlap((const void *)pa[a], t[i].numel * bytes[a], ws, need))
        return FG_EINVAL;
    }
  }
  if (overlap(step_count, 4, ws, need)) return FG_EINVAL;
  return FG_OK;
}

// The flags the update reads may not lie in memory the update writes.
static bool opt_flags_ok(const fg_opt_tensor *t, int32_t n, const int32_t *flags,
                         int32_t nflags, const int32_t *step_count, const void *ws) {
  if (nflags < 0 || (nflags > 0 && !flags)) return false;
  if (nflags == 0) return true;
  const size_t fb = (size_t)nflags * 4;
  if (overlap(flags, fb, step_count, 4) || overlap(flags, fb, ws, lars_adam_ws_bytes(t, n)))
    return false;
  for (int i = 0; i < n; ++i) {
    const uint64_t pa[4] = {t[i].w32, t[i].m, t[i].v, t[i].w16};
    const size_t ba[4] = {4, 4, 4, 2};
    for (int a = 0; a < 4; ++a)
      if (overlap((const void *)pa[a], t[i].numel * ba[a], flags, fb)) return false;
  }
  return true;
}

// Per workspace: which tensors have partial norms for the step in progress
// and which have been applied, for one table, gradient form and set of
// parameters (a hash of them). An apply is accepted only once every tensor
// has norms, and each tensor is applied once; norms are refused while an
// apply is incomplete. A missing or repeated call is thus an error at the
// call instead of a wrong update.
namespace {
struct NormsRecord {
  uint64_t key;
  uint64_t norms;
  uint64_t applied;
};
std::mutex g_norms_mu;
std::unordered_map<uintptr_t, NormsRecord> g_norms;

uint64_t fnv(uint64_t h, const void *p, size_t n) {
  const unsigned char *c = static_cast<const unsigned char *>(p);
  for (size_t i = 0; i < n; ++i) h = (h ^ c[i]) * 0x100000001b3ull;
  return h;
}

uint64_t norms_key(const fg_opt_tensor *t, int32_t n, const fg_opt_params *p,
                   int32_t grad_format, float inv_scale, const int32_t *step_count) {
  uint64_t h = 0xcbf29ce484222325ull;
  h = fnv(h, &n, sizeof n);
  h = fnv(h, t, sizeof(fg_opt_tensor) * (size_t)n);
  const float f[4] = {p->beta1, p->beta2, p->eps, p->weight_decay};
  h = fnv(h, f, sizeof f);
  h = fnv(h, &grad_format, sizeof grad_format);
  const float inv = grad_format == FG_GRAD_F32 ? 0.f : inv_scale;
  h = fnv(h, &inv, sizeof inv);
  const uintptr_t sc = (uintptr_t)step_count;
  return fnv(h, &sc, sizeof sc);
}

uint64_t full_mask(int32_t n) { return n >= 64 ? ~0ull : (1ull << n) - 1; }
}  // namespace

size_t fg_lars_adam_workspace_bytes(const fg_opt_tensor *t, int32_t ntensors) {
  if (!t || ntensors < 1 || ntensors > FG_MAX_SEGMENTS) return 0;
  for (int i = 0; i < ntensors; ++i)
    if (t[i].numel == 0 || t[i].numel >= 0x7FFFFFFFull) return 0;
  return lars_adam_ws_bytes(t, ntensors);
}

fg_status lars_adam_update(const fg_opt_tensor *t, int32_t ntensors,
                           const fg_opt_params *p,
                           const int32_t *found_nonfinite, int32_t nflags,
                           int32_t *step_count, void *ws, size_t ws_bytes,
                           hipStream_t stream) {
  if (nflags < 0 || (nflags > 0 && !found_nonfinite)) return FG_EINVAL;
  const fg_status st =
      opt_call_ok(t, ntensors, p, FG_GRAD_F32, 1.f, step_count, ws, ws_bytes);
  if (st != FG_OK) return st;
  if (!opt_flags_ok(t, ntensors, found_nonfinite, nflags, step_count, ws)) return FG_EINVAL;
  {  // this call overwrites any partial norms held in the workspace
    std::lock_guard<std::mutex> lk(g_norms_mu);
    g_norms.erase((uintptr_t)ws);
  }
  hipError_t e = launch_lars_adam_norms(t, ntensors, 0, ntensors, *p, false, 1.f,
                                        step_count, ws, stream);
  if (e != hipSuccess) return launch_status(e);
  return launch_status(launch_lars_adam_apply(t, ntensors, 0, ntensors, true, *p, false,
                                              1.f, found_nonfinite, nflags, step_count,
                                              ws, stream));
}

fg_status lars_adam_norms(const fg_opt_tensor *t, int32_t ntensors, int32_t first,
                          int32_t count, const fg_opt_params *p, int32_t grad_format,
                          float grad_inv_scale, const int32_t *step_count, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
  const fg_status st =
      opt_call_ok(t, ntensors, p, grad_format, grad_inv_scale, step_count, ws, ws_bytes);
  if (st != FG_OK) return st;
  if (first < 0 || count < 1 || first > ntensors - count) return FG_EINVAL;
  const uint64_t key = norms_key(t, ntensors, p, grad_format, grad_inv_scale, step_count);
  std::lock_guard<std::mutex> lk(g_norms_mu);
  NormsRecord &r = g_norms[(uintptr_t)ws];
  if (r.applied) return FG_EINVAL;  // the previous step's apply is incomplete
  if (r.key != key) r = NormsRecord{key, 0, 0};
  const hipError_t e =
      launch_lars_adam_norms(t, ntensors, first, count, *p,
                             grad_format == FG_GRAD_F16_SCALED, grad_inv_scale,
                             step_count, ws, stream);
  if (e != hipSuccess) return launch_status(e);
  r.norms |= full_mask(first + count) & ~full_mask(first);
  return FG_OK;
}

fg_status lars_adam_apply(const fg_opt_tensor *t, int32_t ntensors, int32_t first,
                          int32_t count, const fg_opt_params *p, int32_t grad_format,
                          float grad_inv_scale, const int32_t *found_nonfinite,
                          int32_t nflags, int32_t *step_count, void *ws,
                          size_t ws_bytes, hipStream_t stream) {
  if (nflags < 0 || (nflags > 0 && !found_nonfinite)) return FG_EINVAL;
  const fg_status st =
      opt_call_ok(t, ntensors, p, grad_format, grad_inv_scale, step_count, ws, ws_bytes);
  if (st != FG_OK) return st;
  if (!opt_flags_ok(t, ntensors, found_nonfinite, nflags, step_count, ws)) return FG_EINVAL;
  if (first < 0 || count < 1 || first > ntensors - count) return FG_EINVAL;
  const uint64_t key = norms_key(t, ntensors, p, grad_format, grad_inv_scale, step_count);
  const uint64_t range = full_mask(first + count) & ~full_mask(first);
  std::lock_guard<std::mutex> lk(g_norms_mu);
  auto it = g_norms.find((uintptr_t)ws);
  if (it == g_norms.end() || it->second.key != key ||
      it->second.norms != full_mask(ntensors) || (it->second.applied & range))
    return FG_EINVAL;
  const hipError_t e = launch_lars_adam_apply(
      t, ntensors, first, count, it->second.applied == 0, *p,
      grad_format == FG_GRAD_F16_SCALED, grad_inv_scale, found_nonfinite, nflags,
      step_count, ws, stream);
  if (e != hipSuccess) return launch_status(e);
  it->second.applied |= range;
  if (it->second.applied == full_mask(ntensors)) g_norms.erase(it);
  return FG_OK;
}

fg_status l2_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                       double scale, uint16_t *dy, hipStream_t stream) {
  if (!y || !t || !dy || numel == 0) return FG_EINVAL;
  if (numel >= (uint64_t)kMaxElems) return FG_EUNSUPPORTED;
  if (overlap(dy, numel * 2, y, numel * 2) || overlap(dy, numel * 2, t, numel * 4))
    return FG_EINVAL;
  return launch_status(launch_head_grad(y, t, numel, scale, dy, stream));
}

// ---- FC-DenseNet variant glue -------------------------------------------
fg_status huber_head_grad(const uint16_t *y, const float *t, uint64_t numel,
                          double scale, double delta, uint16_t *dy,
                          hipStream_t stream) {
  if (!y || !t || !dy || numel == 0) return FG_EINVAL;
  if (!(delta > 0.0) || !std::isfinite(scale)) return FG_EINVAL;
  if (numel >= (uint64_t)kMaxElems) return FG_EUNSUPPORTED;
  if (overlap(dy, numel * 2, y, numel * 2) || overlap(dy, numel * 2, t, numel * 4))
    return FG_EINVAL;
  return launch_status(launch_huber_head_grad(y, t, numel, scale, delta, dy, stream));
}

static fg_status pool_ok(const void *a, const void *b, int32_t n, int32_t h, int32_t w,
                         int32_t c) {
  if (!a || !b || !pos(n) || !pos(h) || !pos(w) || !pos(c)) return FG_EINVAL;
  if (h % 2 || w % 2 || c % 8 || elems4(n, h, w, c) >= kMaxElems) return FG_EUNSUPPORTED;
  if (((uintptr_t)a | (uintptr_t)b) & 15) return FG_EUNSUPPORTED;
  return FG_OK;
}

fg_status avg_pool2d_fwd(const uint16_t *x, int32_t n, int32_t h, int32_t w, int32_t c,
                         uint16_t *y, hipStream_t stream) {
  const fg_status st = pool_ok(x, y, n, h, w, c);
  if (st != FG_OK) return st;
  const size_t big = (size_t)elems4(n, h, w, c) * 2;
  if (overlap(x, big, y, big / 4)) return FG_EINVAL;
  return launch_status(launch_avg_pool2d_fwd(x, n, h, w, c, y, stream));
}

fg_status avg_pool2d_bwd(const uint16_t *dy, const uint16_t *gate, int32_t n, int32_t h,
                         int32_t w, int32_t c, uint16_t *dx, hipStream_t stream) {
  fg_status st = pool_ok(dy, dx, n, h, w, c);
  if (st != FG_OK) return st;
  if (gate && ((uintptr_t)gate & 15)) return FG_EUNSUPPORTED;
  const size_t big = (size_t)elems4(n, h, w, c) * 2;
  if (overlap(dx, big, dy, big / 4) || (gate && overlap(dx, big, gate, big)))
    return FG_EINVAL;
  return launch_status(launch_avg_pool2d_bwd(dy, gate, n, h, w, c, dx, stream));
}

fg_status channel_slice_copy(const uint16_t *src, int32_t src_ld, const uint16_t *gate,
                             int32_t gate_ld, uint16_t *dst, int32_t dst_ld, int64_t npix,
                             int32_t nch, int32_t accumulate, hipStream_t stream) {
  if (!src || !dst || npix <= 0 || !pos(nch) || !pos(src_ld) || !pos(dst_ld) ||
      (gate && !pos(gate_ld)))
    return FG_EINVAL;
  if (nch > src_ld || nch > dst_ld || (gate && nch > gate_ld)) return FG_EINVAL;
  if (nch % 8 || src_ld % 8 || dst_ld % 8 || (gate && gate_ld % 8)) return FG_EUNSUPPORTED;
  if ((((uintptr_t)src | (uintptr_t)dst | (uintptr_t)gate) & 15)) return FG_EUNSUPPORTED;
  const int64_t ld_max = std::max<int64_t>(std::max(src_ld, dst_ld), gate ? gate_ld : 0);
  if (npix * ld_max >= kMaxElems) return FG_EUNSUPPORTED;
  // spans of the three buffers: (npix - 1) * ld + nch elements each
  const size_t ssrc = ((size_t)(npix - 1) * src_ld + nch) * 2;
  const size_t sdst = ((size_t)(npix - 1) * dst_ld + nch) * 2;
  const size_t sgate = gate ? ((size_t)(npix - 1) * gate_ld + nch) * 2 : 0;
  if (overlap(dst, sdst, src, ssrc) || (gate && overlap(dst, sdst, gate, sgate)))
    return FG_EINVAL;
  return launch_status(launch_channel_slice_copy(src, src_ld, gate, gate_ld, dst, dst_ld,
                                                 npix, nch, accumulate != 0, stream));
}

fg_status relu_backward(const uint16_t *dy, const uint16_t *act,
                        uint64_t numel, uint16_t *out, hipStream_t stream) {
  if (!dy || !act || !out || numel == 0) return FG_EINVAL;
  if (numel >= (uint64_t)kMaxElems) return FG_EUNSUPPORTED;
  if (overlap(out, numel * 2, act, numel * 2)) return FG_EINVAL;
  if (out != dy && overlap(out, numel * 2, dy, numel * 2)) return FG_EINVAL;
  return launch_status(launch_relu_backward(dy, act, numel, out, stream));
}

fg_status grad_group_plan(const uint64_t *numel, int32_t ntensors,
                          uint64_t cap_bytes, uint32_t align_bytes,
                          uint32_t elem_bytes, int32_t *group_of,
                          uint64_t *offset_of, int32_t *ngroups,
                          uint64_t *group_numel) {
  if (!numel || ntensors < 1 || !group_of || !offset_of || !ngroups ||
      !group_numel || cap_bytes == 0 || align_bytes == 0 || elem_bytes == 0 ||
      align_bytes % elem_bytes != 0)
    return FG_EINVAL;
  const uint64_t align = align_bytes / elem_bytes;
  int32_t g = 0;
  uint64_t end = 0;
  bool open = false;
  for (int32_t i = 0; i < ntensors; ++i) {
    uint64_t start = (end + align - 1) / align * align;
    if (open && (start + numel[i]) * elem_bytes > cap_bytes) {
      group_numel[g++] = end;
      start = 0;
    }
    group_of[i] = g;
    offset_of[i] = start;
    end = start + numel[i];
    open = true;
  }
  group_numel[g++] = end;
  *ngroups = g;
  return FG_OK;
}

// ---------------------------------------------------------------------------
// Backoff loss scale and learning-rate schedule (host only).
fg_status fg_loss_scale_update(fg_loss_scale *s, int32_t found_nonfinite,
                               int32_t *applied) {
  if (!s || !applied || s->interval < 1 || s->clean < 0 ||
      !(s->s_min > 0.0 && s->s_min <= s->scale && s->scale <= s->s_max) ||
      !std::isfinite(s->s_max))
    return FG_EINVAL;
  if (found_nonfinite) {
    s->scale = std::max(s->scale * 0.5, s->s_min);
    s->clean = 0;
    *applied = 0;
    return FG_OK;
  }
  s->clean += 1;
  if (s->clean >= s->interval) {
    s->scale = std::min(s->scale * 2.0, s->s_max);
    s->clean = 0;
  }
  *applied = 1;
  return FG_OK;
}

fg_status fg_lr_at(const fg_lr_schedule *s, int64_t k, double *lr) {
  if (!s || !lr || k < 0 || !(s->base >= 0.0) || !(s->peak >= 0.0) ||
      s->warmup < 0 || s->every < 0 || !(s->rate > 0.0) || !std::isfinite(s->rate) ||
      !std::isfinite(s->base) || !std::isfinite(s->peak))
    return FG_EINVAL;
  if (k < s->warmup) {
    *lr = s->base + (s->peak - s->base) * (double)k / (double)s->warmup;
    return FG_OK;
  }
  const int64_t steps = s->every ? (k - s->warmup) / s->every : 0;
  *lr = s->peak * std::pow(s->rate, (double)steps);
  return FG_OK;
}

// One-shot profiling events, per host thread (see prof_begin / prof_end).
static thread_local hipEvent_t g_prof_start = nullptr;
static thread_local hipEvent_t g_prof_stop = nullptr;

fg_status fg_mfma_loop(float *out, int32_t blocks, int32_t iters, int32_t operands,
                       hipStream_t stream) {
  if (!out || blocks < 1 || iters < 1 || (operands != 0 && operands != 1) ||
      (int64_t)blocks * iters > FG_MFMA_LOOP_MAX_WORK)
    return FG_EINVAL;
  return launch_status(launch_mfma_loop(out, blocks, iters, operands, stream));
}

fg_status fg_profile_next_launch(hipEvent_t start, hipEvent_t stop) {
  if (!start || !stop) {
    g_prof_start = g_prof_stop = nullptr;
    return FG_OK;
  }
  g_prof_start = start;
  g_prof_stop = stop;
  return FG_OK;
}

}  // extern "C"

namespace fg {
hipError_t prof_begin(hipStream_t st) {
  return g_prof_start ? hipEventRecord(g_prof_start, st) : hipSuccess;
}

hipError_t prof_end(hipStream_t st) {
  if (!g_prof_start) return hipSuccess;
  const hipError_t e = hipEventRecord(g_prof_stop, st);
  g_prof_start = g_prof_stop = nullptr;
  return e;
}
}  // namespace fg
