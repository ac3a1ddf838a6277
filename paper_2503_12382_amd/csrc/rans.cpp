// Host rANS coder for one scale's symbol stream (the paper codes each scale
// independently on the CPU).  Range variant of asymmetric numeral systems
// (Duda, arXiv:1311.2540): 64-bit state kept in [2^31, 2^63), renormalised in
// 32-bit words, 16-bit probability resolution (frequencies sum to 2^16).
// Symbols are pushed in reverse so that decoding pops them in order.

#include <cstdint>
#include <vector>

#include "../../include/reno.h"

namespace {

constexpr uint64_t kLow = uint64_t(1) << 31;  // lower bound of the state interval
constexpr int kProbBits = 16;

// cumulative start of each of the k symbols and the table total (must be 2^16)
bool cumulate(const uint16_t* f, int k, uint32_t* start) {
  uint32_t acc = 0;
  for (int s = 0; s < k; ++s) {
    start[s] = acc;
    acc += f[s];
  }
  start[k] = acc;
  return acc == (1u << kProbBits);
}

// One encoder step: push symbol interval (start, freq) onto state x.
inline void enc_step(uint64_t& x, uint32_t st, uint32_t fs, std::vector<uint32_t>& words) {
  // after the step the state must stay below 2^63: x / fs < 2^(63 - 16)
  const uint64_t bound = (kLow >> kProbBits << 32) * fs;
  while (x >= bound) {
    words.push_back((uint32_t)x);
    x >>= 32;
  }
  x = ((x / fs) << kProbBits) + (x % fs) + st;
}

// Final state and reversal into decode order; false when out is too small.
bool finish(uint64_t x, std::vector<uint32_t>& words, uint32_t* out, int64_t cap, int64_t* nwords) {
  words.push_back((uint32_t)x);
  words.push_back((uint32_t)(x >> 32));
  if ((int64_t)words.size() > cap) return false;
  const size_t m = words.size();
  for (size_t i = 0; i < m; ++i) out[i] = words[m - 1 - i];
  *nwords = (int64_t)m;
  return true;
}

reno_status decode_k(const uint32_t* in, int64_t nwords, const uint16_t* freq, int64_t n, int k,
                     uint8_t* sym) {
  if (!in || (n > 0 && (!freq || !sym)) || n < 0 || (k != 16 && k != 256)) return RENO_E_INVALID;
  if (nwords < 2) return RENO_E_INPUT;
  uint64_t x = ((uint64_t)in[0] << 32) | in[1];
  int64_t pos = 2;
  uint32_t start[257];
  for (int64_t i = 0; i < n; ++i) {
    const uint16_t* f = freq + i * k;
    if (!cumulate(f, k, start)) return RENO_E_INPUT;
    const uint32_t slot = (uint32_t)(x & ((1u << kProbBits) - 1));
    // largest s with start[s] <= slot (binary search over the cumulative table)
    int lo = 0, hi = k;
    while (hi - lo > 1) {
      const int mid = (lo + hi) / 2;
      if (start[mid] <= slot)
        lo = mid;
      else
        hi = mid;
    }
    if (f[lo] == 0) return RENO_E_INPUT;
    sym[i] = (uint8_t)lo;
    x = (uint64_t)f[lo] * (x >> kProbBits) + slot - start[lo];
    while (x < kLow) {
      if (pos >= nwords) return RENO_E_INPUT;
      x = (x << 32) | in[pos++];
    }
  }
  if (pos != nwords || x != kLow) return RENO_E_INPUT;
  return RENO_OK;
}

}  // namespace

extern "C" {

reno_status reno_rans_encode(const uint8_t* sym, const uint16_t* freq, int64_t n, uint32_t* out,
                             int64_t cap, int64_t* nwords_host) {
  if ((n > 0 && (!sym || !freq)) || !out || !nwords_host || n < 0) return RENO_E_INVALID;
  std::vector<uint32_t> words;
  words.reserve((size_t)n / 2 + 4);
  uint32_t start[257];
  uint64_t x = kLow;
  for (int64_t i = n - 1; i >= 0; --i) {
    const uint16_t* f = freq + i * 256;
    if (!cumulate(f, 256, start)) return RENO_E_INPUT;
    const uint32_t fs = f[sym[i]];
    if (fs == 0) return RENO_E_INPUT;
    enc_step(x, start[sym[i]], fs, words);
  }
  return finish(x, words, out, cap, nwords_host) ? RENO_OK : RENO_E_INVALID;
}

reno_status reno_rans_encode_intervals(const uint16_t* iv, int64_t n, int64_t stride, uint32_t* out,
                                       int64_t cap, int64_t* nwords_host) {
  if ((n > 0 && !iv) || !out || !nwords_host || n < 0 || stride < 2) return RENO_E_INVALID;
  std::vector<uint32_t> words;
  words.reserve((size_t)n / 2 + 4);
  uint64_t x = kLow;
  for (int64_t i = n - 1; i >= 0; --i) {
    const uint32_t st = iv[i * stride], fs = iv[i * stride + 1];
    if (fs == 0 || st + fs > (1u << kProbBits)) return RENO_E_INPUT;
    enc_step(x, st, fs, words);
  }
  return finish(x, words, out, cap, nwords_host) ? RENO_OK : RENO_E_INVALID;
}

reno_status reno_rans_decode(const uint32_t* in, int64_t nwords, const uint16_t* freq, int64_t n,
                             uint8_t* sym) {
  return decode_k(in, nwords, freq, n, 256, sym);
}

reno_status reno_rans_decode16(const uint32_t* in, int64_t nwords, const uint16_t* freq, int64_t n,
                               uint8_t* sym) {
  return decode_k(in, nwords, freq, n, 16, sym);
}

}  // extern "C"
