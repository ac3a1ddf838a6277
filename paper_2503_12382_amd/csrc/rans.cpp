// Host rANS coder for one scale's symbol stream (the paper codes each scale
// independently on the CPU).  Range variant of asymmetric numeral systems
// (Duda, arXiv:1311.2540): 64-bit state kept in [2^31, 2^63), renormalised in
// 32-bit words, 16-bit probability resolution (frequencies sum to 2^16).
// Symbols are pushed in reverse so that decoding pops them in order.

#include <algorithm>
#include <atomic>
#include <condition_variable>
#include <cstdint>
#include <functional>
#include <mutex>
#include <thread>
#include <vector>

#include "../../include/reno.h"

namespace {

// Persistent host worker pool for the multi-stream coder: a call hands out
// task indices 0 .. n-1 through an atomic counter to at most `width` threads
// (the caller included) and returns when every task has finished.  Workers
// are created on first use and live until the process ends; calls from
// different host threads are serialised.
class Pool {
 public:
  static Pool& get() {
    static Pool* p = new Pool();  // never destroyed: workers may outlive static destructors
    return *p;
  }

  void run(int n, int width, const std::function<void(int)>& task) {
    std::lock_guard<std::mutex> call(call_mu_);
    width = std::max(1, std::min(width, n));
    grow(width - 1);
    {
      std::lock_guard<std::mutex> lk(mu_);
      task_ = &task;
      n_ = n;
      next_.store(0);
      helpers_ = width - 1;
      busy_ = width - 1;
      ++gen_;
    }
    cv_.notify_all();
    work();
    std::unique_lock<std::mutex> lk(mu_);
    done_cv_.wait(lk, [&] { return busy_ == 0; });
    task_ = nullptr;
  }

 private:
  void grow(int want) {
    while ((int)th_.size() < want) {
      const int id = (int)th_.size();
      th_.emplace_back([this, id] { loop(id); });
      th_.back().detach();
    }
  }

  void work() {
    for (int i = next_.fetch_add(1); i < n_; i = next_.fetch_add(1)) (*task_)(i);
  }

  void loop(int id) {
    uint64_t seen = 0;
    for (;;) {
      {
        std::unique_lock<std::mutex> lk(mu_);
        cv_.wait(lk, [&] { return gen_ != seen; });
        seen = gen_;
        if (id >= helpers_) continue;   // not needed for this call
      }
      work();
      std::lock_guard<std::mutex> lk(mu_);
      if (--busy_ == 0) done_cv_.notify_all();
    }
  }

  std::mutex call_mu_, mu_;
  std::condition_variable cv_, done_cv_;
  std::vector<std::thread> th_;
  const std::function<void(int)>* task_ = nullptr;
  int n_ = 0, helpers_ = 0, busy_ = 0;
  uint64_t gen_ = 0;
  std::atomic<int> next_{0};
};

int pool_width(int threads) {
  if (threads > 0) return std::min(threads, 64);
  const unsigned hc = std::thread::hardware_concurrency();
  return (int)std::max(1u, std::min(hc ? hc : 1u, 16u));
}

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

// Decoding with cumulative tables: start [n][k] holds the start of every
// symbol (start[0] = 0, ascending, the table ends at 2^16), so a symbol is
// found by binary search without summing its table.  Symbols i0, i0 + step,
// ... of the scale; sym is indexed by symbol.
reno_status decode_starts(const uint32_t* in, int64_t nwords, const uint16_t* start, int64_t n, int64_t i0,
                          int64_t step, int k, uint8_t* sym) {
  if (nwords < 2) return RENO_E_INPUT;
  uint64_t x = ((uint64_t)in[0] << 32) | in[1];
  int64_t pos = 2;
  const uint32_t mask = (1u << kProbBits) - 1u;
  for (int64_t i = i0; i < n; i += step) {
    const uint16_t* st = start + i * k;
    const uint32_t slot = (uint32_t)(x & mask);
    int lo = 0, hi = k;  // largest s with st[s] <= slot
    while (hi - lo > 1) {
      const int mid = (lo + hi) / 2;
      if (st[mid] <= slot)
        lo = mid;
      else
        hi = mid;
    }
    const uint32_t a = st[lo], b = lo + 1 < k ? st[lo + 1] : (1u << kProbBits);
    if (st[0] != 0 || b <= a || slot >= b) return RENO_E_INPUT;
    sym[i] = (uint8_t)lo;
    x = (uint64_t)(b - a) * (x >> kProbBits) + slot - a;
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

reno_status reno_rans_encode_streams(const uint16_t* iv, int64_t n, int64_t stride, int nstreams, int threads,
                                     uint32_t* out, int64_t cap, int64_t* nwords_host) {
  if ((n > 0 && !iv) || !out || !nwords_host || n < 0 || stride < 2 || nstreams < 1 ||
      nstreams > RENO_RANS_MAX_STREAMS)
    return RENO_E_INVALID;
  std::vector<std::vector<uint32_t>> words(nstreams);
  std::vector<reno_status> st(nstreams, RENO_OK);
  Pool::get().run(nstreams, pool_width(threads), [&](int j) {
    std::vector<uint32_t>& w = words[j];
    w.reserve((size_t)(n / nstreams) / 2 + 4);
    uint64_t x = kLow;
    const int64_t last = n - 1 - ((n - 1 - j) % nstreams + nstreams) % nstreams;  // last i = j mod S
    for (int64_t i = last; i >= j; i -= nstreams) {
      const uint32_t a = iv[i * stride], f = iv[i * stride + 1];
      if (f == 0 || a + f > (1u << kProbBits)) {
        st[j] = RENO_E_INPUT;
        return;
      }
      enc_step(x, a, f, w);
    }
    w.push_back((uint32_t)x);
    w.push_back((uint32_t)(x >> 32));
    std::reverse(w.begin(), w.end());
  });
  int64_t total = 0;
  for (int j = 0; j < nstreams; ++j) {
    if (st[j] != RENO_OK) return st[j];
    nwords_host[j] = (int64_t)words[j].size();
    total += nwords_host[j];
  }
  if (total > cap) return RENO_E_INVALID;
  int64_t at = 0;
  for (int j = 0; j < nstreams; ++j) {
    std::copy(words[j].begin(), words[j].end(), out + at);
    at += (int64_t)words[j].size();
  }
  return RENO_OK;
}

reno_status reno_rans_decode_streams(const uint32_t* in, const int64_t* nwords_host, int nstreams, int threads,
                                     const uint16_t* start, int k, int64_t n, uint8_t* sym) {
  if (!in || !nwords_host || (n > 0 && (!start || !sym)) || n < 0 || (k != 16 && k != 256) ||
      nstreams < 1 || nstreams > RENO_RANS_MAX_STREAMS)
    return RENO_E_INVALID;
  std::vector<int64_t> off(nstreams + 1, 0);
  for (int j = 0; j < nstreams; ++j) {
    if (nwords_host[j] < 2) return RENO_E_INPUT;
    off[j + 1] = off[j] + nwords_host[j];
  }
  std::vector<reno_status> st(nstreams, RENO_OK);
  Pool::get().run(nstreams, pool_width(threads), [&](int j) {
    st[j] = decode_starts(in + off[j], nwords_host[j], start, n, j, nstreams, k, sym);
  });
  for (int j = 0; j < nstreams; ++j)
    if (st[j] != RENO_OK) return st[j];
  return RENO_OK;
}

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
