// calib.cpp -- host side of the calibration step that precedes the W4Ax path
// (Sec. 3.2): from per-channel maxima of sampled activations, choose the
// outlier channels, a channel permutation that gathers them into the first
// blocks, and the block precision map (8 bits for those blocks, 4 elsewhere).
//
// Rule (the paper fixes the idea, not the constants; both are arguments):
//   med      = lower median of the maxima (rank (K-1)/2 in ascending order);
//   outliers = channels with absmax > ratio * med, compared in fp64 (the
//              product of two floats is exact there); every channel when
//              ratio <= 0, which turns the rule into "fill the cap";
//   n8       = min(ceil(n_out / G), floor(max_frac8 * K/G)) 8-bit blocks;
//   perm     = the n8*G channels ranked first (absmax descending, ties by
//              channel index) in rank order; every later position keeps its
//              own channel unless that channel moved up, and those positions
//              take the channels displaced from the first n8*G positions,
//              ascending to ascending.  Few channels move, so most 8-channel
//              chunks of a row stay in place and the fused gather of the
//              quantizer can read them with one vector load.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <numeric>
#include <vector>

#include "kernels.h"

namespace comet {

const char* plan_channel_perm(const float* absmax, int K, int G, float ratio, float max_frac8,
                              int32_t* perm, uint8_t* prec, int* n_outliers) {
  if (K < 1 || G < 1 || K % G) return "K must be a positive multiple of G";
  if (!(max_frac8 >= 0.0f && max_frac8 <= 1.0f)) return "max_frac8 must lie in [0, 1]";
  if (std::isnan(ratio)) return "outlier_ratio is NaN";
  for (int c = 0; c < K; ++c)
    if (!(absmax[c] >= 0.0f) || std::isinf(absmax[c])) return "absmax holds a negative or non-finite value";
  const int NG = K / G;

  std::vector<float> v(absmax, absmax + K);
  const size_t mid = (size_t)(K - 1) / 2;
  std::nth_element(v.begin(), v.begin() + mid, v.end());
  const double med = v[mid];

  int nout = K;
  if (ratio > 0.0f) {
    const double thr = (double)ratio * med;
    nout = (int)std::count_if(absmax, absmax + K, [&](float a) { return (double)a > thr; });
  }
  const int n8 = std::min((nout + G - 1) / G, (int)std::floor((double)max_frac8 * NG));

  std::vector<int32_t> order(K);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(),
                   [&](int32_t a, int32_t b) { return absmax[a] > absmax[b]; });
  std::vector<uint8_t> in8(K, 0);
  const int head = n8 * G;
  for (int i = 0; i < head; ++i) {
    perm[i] = order[i];
    in8[order[i]] = 1;
  }
  std::vector<int32_t> displaced;
  for (int c = 0; c < head; ++c)
    if (!in8[c]) displaced.push_back(c);
  size_t d = 0;
  for (int p = head; p < K; ++p) perm[p] = in8[p] ? displaced[d++] : p;
  for (int g = 0; g < NG; ++g) prec[g] = g < n8 ? 8 : 4;
  if (n_outliers) *n_outliers = nout;
  return nullptr;
}

}  // namespace comet
