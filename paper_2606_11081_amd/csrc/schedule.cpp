// Host-side learning-rate schedule of App. B "Optimization": warmup over the
// first warmup_frac of the run, starting at start_frac of the peak, then a
// cosine decay to final_frac of the peak.  Linear warmup and a half-cosine
// are the readings taken for the shapes the paper names.
#include <cmath>
#include <cstdint>

#include "gasloc.h"

extern "C" float gasloc_lr_schedule(float peak, int64_t step, int64_t total_steps, float warmup_frac,
                                    float start_frac, float final_frac) {
  const double p = peak, start = start_frac, last = final_frac;
  if (total_steps < 1) return peak;
  const int64_t s = step < 0 ? 0 : (step > total_steps ? total_steps : step);
  const int64_t warm = static_cast<int64_t>(std::floor(static_cast<double>(warmup_frac) *
                                                       static_cast<double>(total_steps)));
  if (s < warm) return static_cast<float>(p * (start + (1.0 - start) * static_cast<double>(s) /
                                                           static_cast<double>(warm)));
  if (warm == total_steps) return peak;
  const double t = static_cast<double>(s - warm) / static_cast<double>(total_steps - warm);
  const double half_cos = (1.0 + std::cos(M_PI * t)) / 2.0;
  return static_cast<float>(p * (last + (1.0 - last) * half_cos));
}
