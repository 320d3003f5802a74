// Offline calibration and export of PRQuant for one alpha (arXiv 2609.22106,
// Algorithm 1 and Eqs. 1-3).  Host-only C++17; compiled without FP contraction
// so every float/double operation rounds exactly as written.
//
//   maxima      a_j = max_t |Xcal[t,j]|, b_j = max_n |W[n,j]|   (Algorithm 1, step 1)
//   scaling     s_j, inv_s_j = 1/s_j, W_s = W diag(s)         (Sec. Method; step 3)
//   selection   column-wise MXFP4 error of W_s, top-k          (step 4)
//   permutation unselected channels, then selected, each ascending   (step 5)
//   residual    R = W~_tail - Q(W~)_tail                        (Eq. 2; step 7)
//   export      Q([W~, R]) packed                               (Eq. 3; step 10)
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <thread>
#include <vector>

#include "prq.h"
#include "prq_internal.h"

namespace {

inline float bf16_to_float(uint16_t h) {
  uint32_t u = static_cast<uint32_t>(h) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// Round a finite float to bf16, nearest with ties to even.
inline uint16_t float_to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}

inline uint32_t float_bits(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  return u;
}

inline float bits_float(uint32_t u) {
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

// E8M0 code of a block from its largest magnitude: the float32 biased exponent
// minus emax(E2M1) = 2, clamped to [0, 254]; 0 for an all-zero block.
inline uint8_t mx_scale_code(float amax) {
  int bexp = static_cast<int>((float_bits(amax) >> 23) & 0xFF);
  int c = bexp - 2;
  return static_cast<uint8_t>(c < 0 ? 0 : (c > 254 ? 254 : c));
}

// 2^(127 - code) as a float; code <= 252 for every finite block, so the
// exponent field 254 - code stays in the normal range.
inline float mx_inv_scale(uint8_t code) { return bits_float(static_cast<uint32_t>(254 - code) << 23); }

// Nearest E2M1 magnitude index of t (|t| < 8), ties to the even index,
// saturating at 6; the sign nibble bit comes from the sign of v (not of t, so
// a value that underflows in the scaling keeps its sign).
inline uint8_t e2m1_code(float t, float v) {
  float a = std::fabs(t);
  int idx = (a > 0.25f) + (a >= 0.75f) + (a > 1.25f) + (a >= 1.75f) + (a > 2.5f) + (a >= 3.5f) +
            (a > 5.0f);
  return static_cast<uint8_t>(idx | ((float_bits(v) >> 31) << 3));
}

const float kE2M1[8] = {0.0f, 0.5f, 1.0f, 1.5f, 2.0f, 3.0f, 4.0f, 6.0f};

inline float e2m1_value(uint8_t code, uint8_t scale) {
  float mag = std::ldexp(kE2M1[code & 7], static_cast<int>(scale) - 127);
  return (code & 8) ? -mag : mag;
}

// Quantize one 32-element block: writes 32 nibbles (unpacked) and returns the scale.
inline uint8_t mx_quantize_block(const float* v, uint8_t* codes) {
  float amax = 0.0f;
  for (int i = 0; i < PRQ_BLOCK; ++i) amax = std::max(amax, std::fabs(v[i]));
  uint8_t sc = mx_scale_code(amax);
  float mul = mx_inv_scale(sc);
  for (int i = 0; i < PRQ_BLOCK; ++i) codes[i] = e2m1_code(v[i] * mul, v[i]);
  return sc;
}

// Quantize one block with a given E8M0 code (code <= 253 keeps 2^(127 - code)
// a normal float); t may reach 16 for code = c0 - 1 and saturates at 6.
inline void mx_quantize_block_with(const float* v, uint8_t sc, uint8_t* codes) {
  float mul = mx_inv_scale(sc);
  for (int i = 0; i < PRQ_BLOCK; ++i) codes[i] = e2m1_code(v[i] * mul, v[i]);
}

// sum_i (v_i - deq_i)^2 in double, one element at a time in index order (each
// difference and square is exact; the order fixes the rounding of the sum).
inline double block_squared_error(const float* v, const uint8_t* codes, uint8_t sc) {
  double err = 0.0;
  for (int i = 0; i < PRQ_BLOCK; ++i) {
    double d = static_cast<double>(v[i]) - static_cast<double>(e2m1_value(codes[i], sc));
    err += d * d;
  }
  return err;
}

// Q(.) with the local E8M0 search of the E8M0-W variant: the first of the
// codes c0, c0 - 1, c0 + 1 (clamped to [0, 254]) with the smallest block error.
inline uint8_t mx_quantize_block_searched(const float* v, uint8_t* codes) {
  uint8_t best = mx_quantize_block(v, codes);
  double best_err = block_squared_error(v, codes, best);
  const int c0 = best;
  uint8_t trial[PRQ_BLOCK];
  for (int off : {-1, 1}) {
    int c = c0 + off;
    c = c < 0 ? 0 : (c > 254 ? 254 : c);
    const uint8_t sc = static_cast<uint8_t>(c);
    mx_quantize_block_with(v, sc, trial);
    const double e = block_squared_error(v, trial, sc);
    if (e < best_err) {
      best_err = e;
      best = sc;
      std::copy(trial, trial + PRQ_BLOCK, codes);
    }
  }
  return best;
}

template <class F>
void parallel_rows(int64_t rows, F&& body) {
  unsigned hw = std::thread::hardware_concurrency();
  int64_t nt = std::max<int64_t>(1, std::min<int64_t>(hw ? hw : 1, 16));
  nt = std::min<int64_t>(nt, std::max<int64_t>(1, rows / 64));
  if (nt <= 1) {
    body(0, rows);
    return;
  }
  std::vector<std::thread> th;
  int64_t per = (rows + nt - 1) / nt;
  for (int64_t t = 0; t < nt; ++t) {
    int64_t r0 = t * per, r1 = std::min(rows, r0 + per);
    if (r0 < r1) th.emplace_back([&body, r0, r1] { body(r0, r1); });
  }
  for (auto& x : th) x.join();
}

}  // namespace

extern "C" int prq_prepare_ex(const uint16_t* W_bf16, int32_t N, int32_t K,
                              const uint16_t* Xcal_bf16, int32_t T, double alpha, int32_t k_tail,
                              int32_t scale_mode, int32_t flags, float* scale, float* inv_scale,
                              int32_t* perm, float* inv_scale_pos, uint8_t* Wq, uint8_t* Wsc,
                              double* col_err) {
  if (!W_bf16 || !Xcal_bf16 || !scale || !inv_scale || !perm || !Wq || !Wsc) return PRQ_EINVAL;
  if (flags & ~PRQ_PREPARE_E8M0_SEARCH) return PRQ_EINVAL;
  const bool search = (flags & PRQ_PREPARE_E8M0_SEARCH) != 0;
  if (N <= 0 || K <= 0 || T <= 0) return PRQ_EINVAL;
  if (!(alpha >= 0.0 && alpha <= 1.0)) return PRQ_EINVAL;
  if (scale_mode != PRQ_SCALE_SMOOTH && scale_mode != PRQ_SCALE_ACT_ONLY &&
      scale_mode != PRQ_SCALE_NONE)
    return PRQ_EINVAL;
  if (K % PRQ_BLOCK || k_tail < 0 || k_tail % PRQ_BLOCK || k_tail > K) return PRQ_EALIGN;
  if (K > 65536) return PRQ_EUNSUPPORTED;
  const int64_t Kaug = static_cast<int64_t>(K) + k_tail;
  const int nb_main = K / PRQ_BLOCK, nb_aug = static_cast<int>(Kaug / PRQ_BLOCK);

  // Algorithm 1, step 1 (and the weight maxima of the smoothing form).
  std::vector<double> a(K, 0.0), b(K, 0.0);
  for (int64_t t = 0; t < T; ++t)
    for (int j = 0; j < K; ++j)
      a[j] = std::max(a[j], static_cast<double>(std::fabs(bf16_to_float(Xcal_bf16[t * K + j]))));
  for (int64_t n = 0; n < N; ++n)
    for (int j = 0; j < K; ++j)
      b[j] = std::max(b[j], static_cast<double>(std::fabs(bf16_to_float(W_bf16[n * K + j]))));

  // Step 3: D_alpha.
  for (int j = 0; j < K; ++j) {
    double aj = std::max(a[j], 1e-5), bj = std::max(b[j], 1e-5);
    double s;
    if (scale_mode == PRQ_SCALE_SMOOTH)
      s = std::pow(aj, alpha) / std::pow(bj, 1.0 - alpha);
    else if (scale_mode == PRQ_SCALE_ACT_ONLY)
      s = std::pow(aj, alpha);
    else
      s = 1.0;
    scale[j] = static_cast<float>(s);
    inv_scale[j] = 1.0f / scale[j];
  }

  // W_s = W D_alpha in float, and its MXFP4 error per column (original order).
  std::vector<float> Ws(static_cast<size_t>(N) * K);
  std::vector<float> E(static_cast<size_t>(N) * K);
  parallel_rows(N, [&](int64_t r0, int64_t r1) {
    std::vector<uint8_t> codes(PRQ_BLOCK);
    for (int64_t n = r0; n < r1; ++n) {
      float* ws = &Ws[n * K];
      float* e = &E[n * K];
      for (int j = 0; j < K; ++j) ws[j] = bf16_to_float(W_bf16[n * K + j]) * scale[j];
      for (int blk = 0; blk < nb_main; ++blk) {
        uint8_t sc = mx_quantize_block(ws + blk * PRQ_BLOCK, codes.data());
        for (int i = 0; i < PRQ_BLOCK; ++i)
          e[blk * PRQ_BLOCK + i] = ws[blk * PRQ_BLOCK + i] - e2m1_value(codes[i], sc);  // exact
      }
    }
  });
  std::vector<double> err(K, 0.0);
  for (int64_t n = 0; n < N; ++n) {  // increasing n, one double add per term
    const float* e = &E[n * K];
    for (int j = 0; j < K; ++j) {
      double d = static_cast<double>(e[j]);
      err[j] += d * d;  // d*d is exact (<= 48 significant bits)
    }
  }
  if (col_err) std::copy(err.begin(), err.end(), col_err);

  // Steps 4-5: top-k (largest error, ties to the smaller index) and the
  // contiguous-tail permutation.
  std::vector<int32_t> order(K);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](int32_t x, int32_t y) {
    return err[x] > err[y] || (err[x] == err[y] && x < y);
  });
  std::vector<char> sel(K, 0);
  for (int i = 0; i < k_tail; ++i) sel[order[i]] = 1;
  int p = 0;
  for (int j = 0; j < K; ++j)
    if (!sel[j]) perm[p++] = j;
  for (int j = 0; j < K; ++j)
    if (sel[j]) perm[p++] = j;
  if (inv_scale_pos)
    for (int q = 0; q < K; ++q) inv_scale_pos[q] = inv_scale[perm[q]];

  // Steps 6, 7, 10: W~ = W_s P, Q(W~), R = W~_tail - Q(W~)_tail, Q(R), packing.
  const int64_t row_bytes = Kaug / 2;
  parallel_rows(N, [&](int64_t r0, int64_t r1) {
    std::vector<float> wt(K), res(k_tail > 0 ? k_tail : 1);
    std::vector<uint8_t> codes(Kaug);
    for (int64_t n = r0; n < r1; ++n) {
      const float* ws = &Ws[n * K];
      for (int q = 0; q < K; ++q) wt[q] = ws[perm[q]];
      uint8_t* sc = Wsc + n * nb_aug;
      for (int blk = 0; blk < nb_main; ++blk)
        sc[blk] = search ? mx_quantize_block_searched(&wt[blk * PRQ_BLOCK], &codes[blk * PRQ_BLOCK])
                         : mx_quantize_block(&wt[blk * PRQ_BLOCK], &codes[blk * PRQ_BLOCK]);
      for (int i = 0; i < k_tail; ++i) {
        int q = K - k_tail + i;
        res[i] = wt[q] - e2m1_value(codes[q], sc[q / PRQ_BLOCK]);  // exact (Eq. 2)
      }
      for (int blk = 0; blk < k_tail / PRQ_BLOCK; ++blk)
        sc[nb_main + blk] =
            search ? mx_quantize_block_searched(&res[blk * PRQ_BLOCK], &codes[K + blk * PRQ_BLOCK])
                   : mx_quantize_block(&res[blk * PRQ_BLOCK], &codes[K + blk * PRQ_BLOCK]);
      uint8_t* out = Wq + n * row_bytes;
      for (int64_t i = 0; i < row_bytes; ++i)
        out[i] = static_cast<uint8_t>(codes[2 * i] | (codes[2 * i + 1] << 4));
    }
  });
  return PRQ_OK;
}

extern "C" int prq_prepare(const uint16_t* W_bf16, int32_t N, int32_t K, const uint16_t* Xcal_bf16,
                           int32_t T, double alpha, int32_t k_tail, int32_t scale_mode,
                           float* scale, float* inv_scale, int32_t* perm,
                           float* inv_scale_pos, uint8_t* Wq, uint8_t* Wsc, double* col_err) {
  return prq_prepare_ex(W_bf16, N, K, Xcal_bf16, T, alpha, k_tail, scale_mode, 0, scale, inv_scale,
                        perm, inv_scale_pos, Wq, Wsc, col_err);
}

extern "C" int prq_expand_producer(const uint16_t* W_up_bf16, const uint16_t* W_gate_bf16, int32_t C,
                                   int32_t H, const float* inv_scale, const int32_t* perm,
                                   int32_t k_tail, uint16_t* W_up_aug, uint16_t* W_gate_aug) {
  if (!W_up_bf16 || !inv_scale || !perm || !W_up_aug || C <= 0 || H <= 0) return PRQ_EINVAL;
  if (W_gate_bf16 && !W_gate_aug) return PRQ_EINVAL;
  if (k_tail < 0 || k_tail > C) return PRQ_EINVAL;
  for (int p = 0; p < C; ++p)
    if (perm[p] < 0 || perm[p] >= C) return PRQ_EINVAL;
  for (int p = 0; p < C; ++p)
    if (!std::isfinite(inv_scale[perm[p]])) return PRQ_EINVAL;
  const int64_t rows = static_cast<int64_t>(C) + k_tail;
  parallel_rows(rows, [&](int64_t r0, int64_t r1) {
    for (int64_t r = r0; r < r1; ++r) {
      // output channel r of the expanded producer: position r (r < C), or the
      // copy of tail position r - k_tail (r >= C)
      const int64_t p = r < C ? r : r - k_tail;
      const int64_t src = perm[p];
      const float d = inv_scale[src];
      const uint16_t* up = W_up_bf16 + src * H;
      uint16_t* out = W_up_aug + r * H;
      for (int h = 0; h < H; ++h) out[h] = float_to_bf16(bf16_to_float(up[h]) * d);
      if (W_gate_bf16)
        std::memcpy(W_gate_aug + r * H, W_gate_bf16 + src * H, static_cast<size_t>(H) * 2);
    }
  });
  return PRQ_OK;
}
