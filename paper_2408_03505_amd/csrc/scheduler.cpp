// Kernel-to-bubble packing (the ScheduleKernels step of the bubble
// scheduler, §4.2): the encoder's kernels, in chain order, go into the LLM
// timeline -- computation kernels into bubbles, several per bubble while
// their summed time fits, communication kernels into periods of LLM
// computation (§3.1, design decision 3) -- each into the earliest interval
// of its kind, at or after its predecessor's, that still holds it.
// Host code; no GPU is involved.
#include <math.h>

#include "../../include/optimus_enc.h"
#include "status.hpp"

using optimus::clear_error;
using optimus::set_error;

extern "C" int enc_schedule_kernels(const double *kernel_us, const int *kernel_comm, int n_kernels,
                                    const double *interval_us, const int *interval_bubble, int n_intervals,
                                    int *out_interval, double *out_offset_us) {
  const char *fn = "enc_schedule_kernels";
  if (n_kernels < 0 || n_intervals < 0) return set_error(ENC_ERR_INVALID, "%s: counts must be >= 0", fn);
  if (n_kernels > 0 && (!kernel_us || !out_interval))
    return set_error(ENC_ERR_INVALID, "%s: kernel_us and out_interval must not be NULL", fn);
  if (n_intervals > 0 && (!interval_us || !interval_bubble))
    return set_error(ENC_ERR_INVALID, "%s: interval_us and interval_bubble must not be NULL", fn);
  for (int i = 0; i < n_kernels; ++i)
    if (!(kernel_us[i] >= 0.0) || isinf(kernel_us[i]))
      return set_error(ENC_ERR_INVALID, "%s: kernel_us[%d] must be finite and >= 0", fn, i);
  for (int j = 0; j < n_intervals; ++j)
    if (!(interval_us[j] >= 0.0) || isinf(interval_us[j]))
      return set_error(ENC_ERR_INVALID, "%s: interval_us[%d] must be finite and >= 0", fn, j);

  for (int i = 0; i < n_kernels; ++i) {
    out_interval[i] = -1;
    if (out_offset_us) out_offset_us[i] = -1.0;
  }
  int cur = 0;        // interval of the previous kernel
  double used = 0.0;  // time already taken in interval `cur`
  int placed = 0;
  for (int i = 0; i < n_kernels; ++i) {
    const double d = kernel_us[i];
    const bool wants_bubble = !(kernel_comm && kernel_comm[i]);
    int where = -1;
    double start = 0.0;
    for (int j = cur; j < n_intervals; ++j) {
      if ((interval_bubble[j] != 0) != wants_bubble) continue;
      const double s = (j == cur) ? used : 0.0;
      if (s + d <= interval_us[j]) {
        where = j;
        start = s;
        break;
      }
    }
    if (where < 0) break;  // this kernel and every later one stay unplaced
    out_interval[i] = where;
    if (out_offset_us) out_offset_us[i] = start;
    cur = where;
    used = start + d;
    ++placed;
  }
  clear_error();
  return placed;
}
