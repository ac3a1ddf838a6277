// Whole-frame coding: one frame's geometry to a self-describing bitstream and
// back (the codec of Sec. 3 with the entropy coder of Sec. 4.2), every step
// on the GPU.  The encoder runs the pyramid, the model on every scale, the
// symbol intervals and the rANS streams (k_code.hip) and copies the finished
// bitstream out once.  The decoder copies the bitstream in once and enqueues
// the whole per-scale chain (expand, predict, cumulative tables, stream
// decoding into the next scale's codes) without waiting on the host; it
// synchronises only at the end, where device-side checks are reported.
// Staging buffers belong to the context and grow on demand.
//
// Bitstream (uint32 words): 0x4F4E4552 ("RENO" as little-endian bytes), B,
// b0, stages, L, N_b0; the base voxels bit-packed from the lowest bit up as
// fields x | y << b0 | z << 2 b0 | code << 3 b0 of 3 b0 + 8 bits; then one
// section per model scale b0 < b < B and stage: S = ceil(N_b / L) stream
// lengths (16 bits each, two per word, the even stream in the low half; an
// empty scale has one empty stream) followed by the S streams, stream j
// holding symbols j, j + S, ... as a single-stream rANS code.

#include <algorithm>
#include <cstring>
#include <string>

#include "ctx.h"

namespace reno {
namespace {

constexpr uint32_t kMagic = 0x4F4E4552u;
constexpr int kHeader = 6;
constexpr int kMaxStreamSymbols = 65533;  // stream lengths (L + 2 words at most) fit 16 bits

enum { D_WORDS, D_REGION, D_BOOK, D_TAB, D_BASE };  // device staging
enum { H_WORDS, H_AUX };                             // pinned host staging

reno_status frame_fail(Ctx* c, reno_status s, const std::string& msg) {
  c->err = msg;
  return s;
}

#define FRAME_HIP(c, expr)                                                                      \
  do {                                                                                          \
    hipError_t e_ = (expr);                                                                     \
    if (e_ != hipSuccess)                                                                       \
      return frame_fail((c), RENO_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));    \
  } while (0)

#define FRAME_OK(expr)            \
  do {                            \
    reno_status s_ = (expr);      \
    if (s_ != RENO_OK) return s_; \
  } while (0)

size_t round_up(size_t n) { return (std::max<size_t>(n, 1) + 4095) & ~size_t(4095); }

hipError_t dev_buf(Ctx& c, int i, size_t bytes) {
  if (c.fc_dev_bytes[i] >= bytes) return hipSuccess;
  if (c.fc_dev[i]) (void)hipFree(c.fc_dev[i]);
  c.fc_dev[i] = nullptr;
  c.fc_dev_bytes[i] = 0;
  const size_t n = round_up(bytes);
  hipError_t e = hipMalloc(&c.fc_dev[i], n);
  if (e == hipSuccess) c.fc_dev_bytes[i] = n;
  return e;
}

hipError_t host_buf(Ctx& c, int i, size_t bytes) {
  if (c.fc_host_bytes[i] >= bytes) return hipSuccess;
  if (c.fc_host[i]) (void)hipHostFree(c.fc_host[i]);
  c.fc_host[i] = nullptr;
  c.fc_host_bytes[i] = 0;
  const size_t n = round_up(bytes);
  hipError_t e = hipHostMalloc(&c.fc_host[i], n, 0);
  if (e == hipSuccess) c.fc_host_bytes[i] = n;
  return e;
}

int64_t base_words(int64_t n0, int b0) { return (n0 * (3 * b0 + 8) + 31) / 32; }

// Once a call has enqueued work (kernels, copies through the pinned staging
// buffers), an early return still waits for its stream, so that the next
// call never refills a staging buffer that a copy is still reading.
struct DrainOnExit {
  Ctx* c;
  bool armed = false;
  ~DrainOnExit() {
    if (armed) (void)hipStreamSynchronize(c->stream);
  }
};

}  // namespace

void frame_free(Ctx& c) {
  for (int i = 0; i < Ctx::FC_DEV; ++i) {
    if (c.fc_dev[i]) (void)hipFree(c.fc_dev[i]);
    c.fc_dev[i] = nullptr;
    c.fc_dev_bytes[i] = 0;
  }
  for (int i = 0; i < Ctx::FC_HOST; ++i) {
    if (c.fc_host[i]) (void)hipHostFree(c.fc_host[i]);
    c.fc_host[i] = nullptr;
    c.fc_host_bytes[i] = 0;
  }
}

}  // namespace reno

extern "C" {

reno_status reno_encode_frame(reno_ctx* c, const float* points, int64_t n, int bit_depth, int stream_symbols,
                              uint32_t* out_host, int64_t cap_words, int64_t* nwords_host) {
  using namespace reno;
  if (!c) return RENO_E_INVALID;
  if (!nwords_host || cap_words < 0 || (cap_words > 0 && !out_host))
    return frame_fail(c, RENO_E_INVALID, "null or negative output");
  const int L = stream_symbols;
  if (L < 1 || L > kMaxStreamSymbols) return frame_fail(c, RENO_E_INVALID, "stream_symbols must be in [1, 65533]");
  const int b0 = c->b0();
  if (3 * b0 + 8 > 32) return frame_fail(c, RENO_E_INVALID, "frame coding needs min_bit_depth <= 8");
  if (!c->have_weights) return frame_fail(c, RENO_E_STATE, "no weights set");
  DrainOnExit drain{c};
  drain.armed = true;
  FRAME_OK(reno_build_pyramid(c, points, n, bit_depth));
  FRAME_OK(reno_predict_probs(c, RENO_ALL_SCALES, nullptr, nullptr));
  const int B = bit_depth;
  const int stages = c->p.head_mode == RENO_HEAD_TWO_STAGE ? 2 : 1;
  const int sections = (B - 1 - b0) * stages;
  const int64_t G = sections > 0 ? rans_stream_bound(*c, sections, L) : 0;
  const int64_t n0_max = std::min<int64_t>(c->cap_pts, int64_t(1) << (3 * b0));
  const int64_t cap_dev = kHeader + base_words(n0_max, b0) + G + sections + G * (int64_t)(L + 2);
  FRAME_HIP(c, dev_buf(*c, D_WORDS, sizeof(uint32_t) * (size_t)cap_dev));
  FRAME_HIP(c, dev_buf(*c, D_REGION, sizeof(uint32_t) * (size_t)G * (L + 2)));
  FRAME_HIP(c, dev_buf(*c, D_BOOK, (sizeof(uint32_t) + sizeof(int64_t)) * (size_t)G + 64));
  FRAME_HIP(c, dev_buf(*c, D_TAB, sizeof(uint16_t) * 2 * stages * (size_t)c->cap_model));
  FRAME_HIP(c, dev_buf(*c, D_BASE, sizeof(int32_t) * 3 * (size_t)c->cap_pts));
  FRAME_HIP(c, host_buf(*c, H_AUX, 64));
  uint32_t* words = static_cast<uint32_t*>(c->fc_dev[D_WORDS]);
  uint32_t* region = static_cast<uint32_t*>(c->fc_dev[D_REGION]);
  int64_t* total = static_cast<int64_t*>(c->fc_dev[D_BOOK]);  // [0] words, [1] streams
  int64_t* offs = total + 8;
  uint32_t* lens = reinterpret_cast<uint32_t*>(offs + G);
  uint16_t* iv = static_cast<uint16_t*>(c->fc_dev[D_TAB]);
  int32_t* xyz = static_cast<int32_t*>(c->fc_dev[D_BASE]);
  if (sections > 0) {
    FRAME_OK(reno_symbol_intervals(c, RENO_ALL_SCALES, iv));
    FRAME_HIP(c, launch_rans_encode(*c, iv, b0 + 1, B - 1, stages, L, region, lens, G));
  }
  FRAME_OK(reno_coords(c, b0, xyz, nullptr));
  FRAME_HIP(c, launch_rans_layout(*c, b0 + 1, B - 1, stages, L, B, lens, G, offs, words, cap_dev, total));
  FRAME_HIP(c, launch_rans_pack(*c, region, lens, offs, L, G, total, xyz, words, cap_dev));
  int64_t* tot_host = static_cast<int64_t*>(c->fc_host[H_AUX]);
  FRAME_HIP(c, hipMemcpyAsync(tot_host, total, 2 * sizeof(int64_t), hipMemcpyDeviceToHost, c->stream));
  FRAME_OK(reno_sync(c));
  drain.armed = false;  // reno_sync waited for the stream
  const int64_t nw = tot_host[0];
  *nwords_host = nw;
  if (nw > cap_words) return frame_fail(c, RENO_E_CAPACITY, "bitstream exceeds cap_words");
  FRAME_HIP(c, host_buf(*c, H_WORDS, sizeof(uint32_t) * (size_t)nw));
  drain.armed = true;
  FRAME_HIP(c, hipMemcpyAsync(c->fc_host[H_WORDS], words, sizeof(uint32_t) * (size_t)nw, hipMemcpyDeviceToHost,
                              c->stream));
  FRAME_HIP(c, hipStreamSynchronize(c->stream));
  drain.armed = false;
  std::memcpy(out_host, c->fc_host[H_WORDS], sizeof(uint32_t) * (size_t)nw);
  return RENO_OK;
}

reno_status reno_decode_frame(reno_ctx* c, const uint32_t* in_host, int64_t nwords) {
  using namespace reno;
  if (!c) return RENO_E_INVALID;
  if (!in_host || nwords < kHeader) return frame_fail(c, RENO_E_INPUT, "bitstream shorter than its header");
  if (!c->have_weights) return frame_fail(c, RENO_E_STATE, "no weights set");
  const bool two = c->p.head_mode == RENO_HEAD_TWO_STAGE;
  const int stages = two ? 2 : 1;
  const int b0 = c->b0();
  const int64_t B = in_host[1], L = in_host[4], n0 = in_host[5];
  if (in_host[0] != kMagic) return frame_fail(c, RENO_E_INPUT, "not a frame bitstream");
  if ((int64_t)in_host[2] != b0) return frame_fail(c, RENO_E_INPUT, "min_bit_depth differs from the context's");
  if (3 * b0 + 8 > 32) return frame_fail(c, RENO_E_INVALID, "frame coding needs min_bit_depth <= 8");
  if (B <= b0 || B > c->p.max_bit_depth) return frame_fail(c, RENO_E_INPUT, "bit depth out of range");
  if ((int64_t)in_host[3] != stages) return frame_fail(c, RENO_E_INPUT, "head stages differ from the context's");
  if (L < 1 || L > kMaxStreamSymbols) return frame_fail(c, RENO_E_INPUT, "stream length out of range");
  if (n0 > std::min<int64_t>(c->cap_pts, int64_t(1) << (3 * b0)))
    return frame_fail(c, RENO_E_INPUT, "base count out of range");
  const int64_t p0 = kHeader + base_words(n0, b0);
  const int sections = (int)(B - 1 - b0) * stages;
  if (p0 > nwords || (sections == 0 && p0 != nwords))
    return frame_fail(c, RENO_E_INPUT, "bitstream length does not match its base voxels");
  const int K = two ? 16 : 256;
  FRAME_HIP(c, dev_buf(*c, D_WORDS, sizeof(uint32_t) * (size_t)nwords));
  FRAME_HIP(c, host_buf(*c, H_WORDS, sizeof(uint32_t) * (size_t)nwords));
  FRAME_HIP(c, dev_buf(*c, D_BOOK, sizeof(uint64_t) * (size_t)(sections + 1)));
  // the decoder's entries (uint32 per symbol), then room for the uint16
  // cumulative tables that contexts outside the register-resident table
  // kernels pass through
  FRAME_HIP(c, dev_buf(*c, D_TAB, (sizeof(uint32_t) + sizeof(uint16_t)) * (size_t)K * c->cap_pts));
  FRAME_HIP(c, dev_buf(*c, D_BASE, (sizeof(int32_t) * 3 + 3) * (size_t)c->cap_pts));
  FRAME_HIP(c, host_buf(*c, H_AUX, (sizeof(int32_t) * 3 + 1) * (size_t)std::max<int64_t>(n0, 1)));
  // base voxels, unpacked on the host (the header is read there anyway)
  int32_t* xyz_h = static_cast<int32_t*>(c->fc_host[H_AUX]);
  uint8_t* code_h = reinterpret_cast<uint8_t*>(xyz_h + 3 * std::max<int64_t>(n0, 1));
  {
    const int wd = 3 * b0 + 8;
    const uint32_t* src = in_host + kHeader;
    const uint64_t fmask = (uint64_t(1) << wd) - 1;
    const uint32_t m = (1u << b0) - 1u;
    for (int64_t v = 0; v < n0; ++v) {
      const int64_t bit = v * wd, q = bit / 32, r = bit % 32;
      uint64_t f = src[q] >> r;
      if (r + wd > 32) f |= (uint64_t)src[q + 1] << (32 - r);
      f &= fmask;
      xyz_h[3 * v] = (int32_t)(f & m);
      xyz_h[3 * v + 1] = (int32_t)((f >> b0) & m);
      xyz_h[3 * v + 2] = (int32_t)((f >> (2 * b0)) & m);
      code_h[v] = (uint8_t)(f >> (3 * b0));
      if (code_h[v] == 0) return frame_fail(c, RENO_E_INPUT, "a base occupancy code is zero");
    }
  }
  int32_t* xyz_d = static_cast<int32_t*>(c->fc_dev[D_BASE]);
  uint8_t* base_code_d = reinterpret_cast<uint8_t*>(xyz_d + 3 * c->cap_pts);
  uint8_t* code_d = base_code_d + c->cap_pts;
  uint8_t* s1_d = code_d + c->cap_pts;
  uint32_t* words_d = static_cast<uint32_t*>(c->fc_dev[D_WORDS]);
  uint64_t* fpos = static_cast<uint64_t*>(c->fc_dev[D_BOOK]);
  uint32_t* tab = static_cast<uint32_t*>(c->fc_dev[D_TAB]);
  uint16_t* tab_scratch = reinterpret_cast<uint16_t*>(tab + (size_t)K * c->cap_pts);
  std::memcpy(c->fc_host[H_WORDS], in_host, sizeof(uint32_t) * (size_t)nwords);
  DrainOnExit drain{c};
  drain.armed = true;
  FRAME_HIP(c, hipMemcpyAsync(words_d, c->fc_host[H_WORDS], sizeof(uint32_t) * (size_t)nwords,
                              hipMemcpyHostToDevice, c->stream));
  if (n0 > 0) {
    FRAME_HIP(c, hipMemcpyAsync(xyz_d, xyz_h, sizeof(int32_t) * 3 * (size_t)n0, hipMemcpyHostToDevice, c->stream));
    FRAME_HIP(c, hipMemcpyAsync(base_code_d, code_h, (size_t)n0, hipMemcpyHostToDevice, c->stream));
  }
  FRAME_OK(reno_set_base(c, (int)B, xyz_d, base_code_d, n0));
  const uint8_t* prev = nullptr;  // codes of the scale below (the base scale's are recorded by set_base)
  int t = 0;
  for (int b = b0 + 1; b < B; ++b) {
    FRAME_OK(reno_expand(c, b - 1, prev));
    FRAME_OK(reno_predict_probs(c, b, nullptr, nullptr));
    if (two) {
      FRAME_HIP(c, launch_symbol_entries(*c, b, 1, tab, tab_scratch));
      FRAME_HIP(c, launch_rans_decode(*c, words_d, nwords, b, (int)L, K, tab, nullptr, s1_d, fpos, t, p0,
                                      t == sections - 1));
      ++t;
      FRAME_OK(reno_predict_second(c, b, s1_d, nullptr));
      FRAME_HIP(c, launch_symbol_entries(*c, b, 2, tab, tab_scratch));
      FRAME_HIP(c, launch_rans_decode(*c, words_d, nwords, b, (int)L, K, tab, s1_d, code_d, fpos, t, p0,
                                      t == sections - 1));
      ++t;
    } else {
      FRAME_HIP(c, launch_symbol_entries(*c, b, 0, tab, tab_scratch));
      FRAME_HIP(c, launch_rans_decode(*c, words_d, nwords, b, (int)L, K, tab, nullptr, code_d, fpos, t, p0,
                                      t == sections - 1));
      ++t;
    }
    prev = code_d;
  }
  FRAME_OK(reno_expand(c, (int)B - 1, prev));
  const reno_status st = reno_sync(c);
  drain.armed = false;  // the stream has been waited for
  return st;
}

}  // extern "C"
