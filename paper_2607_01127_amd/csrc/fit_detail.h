// Private interface between the device fit's kernels (logbq_kernels.hip) and its exact host-side
// selection (fit.cpp). Not part of the public ABI.
//
// The device fit finds w_min of Eq. 5 (Sec. 3.2) by a radix selection over the float32 bit
// patterns of |w| (sign cleared; for finite values their integer order is their value order).
// Pass 1 bins bits 30..20 of every pattern (2048 bins). Pass 2 bins bits 19..11 of the patterns
// whose bits 30..20 equal the bin chosen in pass 1 (512 bins). Pass 3 bins bits 10..0 of the
// patterns whose bits 30..11 equal the choice so far (2048 bins), so its bins are single values.
// Bits 30..23 are the exponent field, so all weights of one bin share an exponent, and the
// energy of a bin is an integer sum of squared significands times one power of two.
#pragma once

#include <cstdint>

#include "logbq.h"

namespace logbq_detail {

constexpr int kFitBins1 = 2048;   // bins of pass 1
constexpr int kFitBins2 = 512;    // bins of pass 2
constexpr int kFitBins3 = 2048;   // bins of pass 3

// One pass's result on the host. bins holds three unsigned 64-bit words per bin: the number of
// weights, the sum of (m^2 >> 24) and the sum of (m^2 & 0xFFFFFF), where m is the integer
// significand of |w| (24 bits with the implicit bit; the 23 stored bits for subnormals).
struct FitPassResult {
  const uint64_t* bins;
  uint32_t max_key;     // pass 1: largest bit pattern of |w|
  uint32_t nonfinite;   // pass 1: nonzero if some weight is NaN or Inf
};

// Runs pass `pass` (1, 2 or 3) over the weights with the selection `sel` (pass 2: the pass-1
// bin; pass 3: bits 30..11) and fills *res; returns a logbq status.
typedef int32_t (*FitPassFn)(void* ctx, int pass, uint32_t sel, FitPassResult* res);

// Eq. 5 with exact sums: w_min is |w| at the smallest position i of |w| sorted ascending whose
// exact prefix energy sum_{j <= i} w_j^2 reaches eps times the exact total. Then b, s, the
// codebook and the thresholds exactly as logbq_fit computes them from w_min, w_max and i.
// Errors as logbq_fit: NONFINITE, DEGENERATE; HIP if the passes' bins are inconsistent.
int32_t fit_from_passes(int32_t bits, double eps, FitPassFn run, void* ctx, logbq_params* out);

}  // namespace logbq_detail
