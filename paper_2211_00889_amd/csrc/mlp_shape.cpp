// Host checks of the end-to-end MLP workload's shape (plain C++, no HIP): the
// supported shapes, the flat parameter layout and the workspace size.
#include "mlp_shape.h"

#include "internal.h"

namespace nbsgd {

nbsgd_status check_shape(const nbsgd_mlp_shape* s, Dims* d) {
  if (!s) return fail(NBSGD_E_ARG, "shape is null");
  if (s->batch != kBatch)
    return fail(NBSGD_E_UNSUPPORTED, "batch=%d: only %d is supported", s->batch, kBatch);
  if (s->d_in < kFeatBlock || s->d_in % kFeatBlock || s->hidden < 64 || s->hidden % 64 ||
      s->hidden > kMaxHidden)
    return fail(NBSGD_E_UNSUPPORTED,
                "d_in=%d must be a multiple of %d and hidden=%d a multiple of 64, at most %d",
                s->d_in, kFeatBlock, s->hidden, kMaxHidden);
  if (s->classes < 2 || s->classes > kMaxClasses)
    return fail(NBSGD_E_UNSUPPORTED, "classes=%d must be in [2, %d]", s->classes, kMaxClasses);
  // flat layout: W1[d_in][hidden], b1[hidden], W2[hidden][classes],
  // b2[classes], zeros up to a multiple of 4 floats
  d->d_in = s->d_in;
  d->hidden = s->hidden;
  d->classes = s->classes;
  d->off_b1 = (int64_t)s->d_in * s->hidden;
  d->off_w2 = d->off_b1 + s->hidden;
  d->off_b2 = d->off_w2 + (int64_t)s->hidden * s->classes;
  d->off_pad = d->off_b2 + s->classes;
  d->P = (d->off_pad + 3) & ~(int64_t)3;
  d->ld = d->P;
  return NBSGD_OK;
}

}  // namespace nbsgd

using namespace nbsgd;

extern "C" nbsgd_status nbsgd_mlp_param_count(const nbsgd_mlp_shape* s, int64_t* P) {
  clear_error();
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (!P) return fail(NBSGD_E_ARG, "P is null");
  *P = d.P;
  return NBSGD_OK;
}

extern "C" nbsgd_status nbsgd_mlp_workspace_bytes(const nbsgd_mlp_shape* s, int64_t rows,
                                                  size_t* bytes) {
  clear_error();
  Dims d;
  if (nbsgd_status st = check_shape(s, &d)) return st;
  if (!bytes || rows < 0) return fail(NBSGD_E_ARG, "bytes is null or rows < 0");
  *bytes = workspace_for(d, rows);
  return NBSGD_OK;
}
