// Whole-frame coding: one frame's geometry to a self-describing bitstream and
// back (the codec of Sec. 3 with the arithmetic coder of Sec. 4.2 on the
// host).  The encoder runs the pyramid, the model on every scale and the
// symbol intervals on the GPU, then codes every scale (and stage) as
// interleaved rANS streams on the library's host thread pool.  The decoder
// drives the per-scale loop natively: expand the previous scale, predict,
// copy the cumulative tables out, decode the scale's streams on the host,
// copy the codes back in.  Staging buffers (device and pinned host) belong to
// the context and grow on demand.
//
// Bitstream (uint32 words): "RENO" magic, B, b0, stages, S, N_b0; the base
// voxels bit-packed as (x, y, z, code) fields of 3 b0 + 8 bits, low bits
// first; then for every model scale b0 < b < B and every stage, the S word
// counts followed by the S streams (stream j holds symbols j, j + S, ...).

#include <algorithm>
#include <string>
#include <vector>

#include "ctx.h"

namespace reno {
namespace {

constexpr uint32_t kMagic = 0x4F4E4552u;  // "RENO" read as little-endian bytes
constexpr int kHeader = 6;

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

#define FRAME_OK(expr)                 \
  do {                                 \
    reno_status s_ = (expr);           \
    if (s_ != RENO_OK) return s_;      \
  } while (0)

// device + pinned host buffer of at least `bytes`, grown on demand
hipError_t grow(void** dev, void** host, size_t* have, size_t bytes) {
  if (*have >= bytes) return hipSuccess;
  if (*dev) (void)hipFree(*dev);
  if (*host) (void)hipHostFree(*host);
  *dev = *host = nullptr;
  *have = 0;
  const size_t n = (bytes + 4095) & ~size_t(4095);
  hipError_t e = hipMalloc(dev, n);
  if (e != hipSuccess) return e;
  e = hipHostMalloc(host, n, 0);
  if (e != hipSuccess) return e;
  *have = n;
  return hipSuccess;
}

// little-endian bit writer / reader over uint32 words
struct BitWriter {
  std::vector<uint32_t>& out;
  uint64_t acc = 0;
  int nbits = 0;
  void put(uint32_t v, int w) {
    acc |= (uint64_t)v << nbits;
    nbits += w;
    while (nbits >= 32) {
      out.push_back((uint32_t)acc);
      acc >>= 32;
      nbits -= 32;
    }
  }
  void flush() {
    if (nbits > 0) out.push_back((uint32_t)acc);
    acc = 0;
    nbits = 0;
  }
};

struct BitReader {
  const uint32_t* in;
  int64_t n, pos = 0;
  uint64_t acc = 0;
  int nbits = 0;
  bool get(int w, uint32_t* v) {
    while (nbits < w) {
      if (pos >= n) return false;
      acc |= (uint64_t)in[pos++] << nbits;
      nbits += 32;
    }
    *v = (uint32_t)(acc & ((uint64_t(1) << w) - 1));
    acc >>= w;
    nbits -= w;
    return true;
  }
};

}  // namespace

void frame_free(Ctx& c) {
  if (c.fc_tab_dev) (void)hipFree(c.fc_tab_dev);
  if (c.fc_tab_host) (void)hipHostFree(c.fc_tab_host);
  if (c.fc_aux_dev) (void)hipFree(c.fc_aux_dev);
  if (c.fc_aux_host) (void)hipHostFree(c.fc_aux_host);
  c.fc_tab_dev = c.fc_tab_host = c.fc_aux_dev = c.fc_aux_host = nullptr;
  c.fc_tab_bytes = c.fc_aux_bytes = 0;
}

}  // namespace reno

extern "C" {

reno_status reno_encode_frame(reno_ctx* c, const float* points, int64_t n, int bit_depth, int nstreams,
                              uint32_t* out_host, int64_t cap_words, int64_t* nwords_host) {
  using namespace reno;
  if (!c) return RENO_E_INVALID;
  if (!out_host || !nwords_host) return frame_fail(c, RENO_E_INVALID, "null output");
  if (nstreams < 1 || nstreams > RENO_RANS_MAX_STREAMS)
    return frame_fail(c, RENO_E_INVALID, "nstreams must be in [1, RENO_RANS_MAX_STREAMS]");
  const int b0 = c->b0();
  if (3 * b0 + 8 > 32) return frame_fail(c, RENO_E_INVALID, "frame coding needs min_bit_depth <= 8");
  if (!c->have_weights) return frame_fail(c, RENO_E_STATE, "no weights set");
  FRAME_OK(reno_build_pyramid(c, points, n, bit_depth));
  const int B = bit_depth;
  const bool two = c->p.head_mode == RENO_HEAD_TWO_STAGE;
  const int per = two ? 4 : 2, stages = two ? 2 : 1;
  FRAME_OK(reno_predict_probs(c, RENO_ALL_SCALES, nullptr, nullptr));
  int64_t counts[NLEV];
  FRAME_OK(reno_scale_counts(c, counts));  // synchronises: the sizes below are exact
  int64_t nm = 0;
  for (int b = b0 + 1; b < B; ++b) nm += counts[b];
  const int64_t n0 = counts[b0];
  FRAME_HIP(c, grow(&c->fc_tab_dev, &c->fc_tab_host, &c->fc_tab_bytes,
                    sizeof(uint16_t) * (size_t)std::max<int64_t>(nm, 1) * per));
  FRAME_HIP(c, grow(&c->fc_aux_dev, &c->fc_aux_host, &c->fc_aux_bytes,
                    (sizeof(int32_t) * 3 + 2) * (size_t)std::max<int64_t>(n0, 1)));
  uint16_t* iv_dev = static_cast<uint16_t*>(c->fc_tab_dev);
  int32_t* xyz_dev = static_cast<int32_t*>(c->fc_aux_dev);
  uint8_t* code_dev = reinterpret_cast<uint8_t*>(xyz_dev + 3 * std::max<int64_t>(n0, 1));
  if (nm > 0) FRAME_OK(reno_symbol_intervals(c, RENO_ALL_SCALES, iv_dev));
  FRAME_OK(reno_coords(c, b0, xyz_dev, nullptr));
  FRAME_OK(reno_occupancy_codes(c, b0, code_dev));
  const size_t xyz_off = reinterpret_cast<char*>(xyz_dev) - static_cast<char*>(c->fc_aux_dev);
  const size_t code_off = reinterpret_cast<char*>(code_dev) - static_cast<char*>(c->fc_aux_dev);
  if (nm > 0)
    FRAME_HIP(c, hipMemcpyAsync(c->fc_tab_host, iv_dev, sizeof(uint16_t) * (size_t)nm * per,
                                hipMemcpyDeviceToHost, c->stream));
  if (n0 > 0) {
    FRAME_HIP(c, hipMemcpyAsync(static_cast<char*>(c->fc_aux_host) + xyz_off, xyz_dev,
                                sizeof(int32_t) * 3 * (size_t)n0, hipMemcpyDeviceToHost, c->stream));
    FRAME_HIP(c, hipMemcpyAsync(static_cast<char*>(c->fc_aux_host) + code_off, code_dev, (size_t)n0,
                                hipMemcpyDeviceToHost, c->stream));
  }
  FRAME_OK(reno_sync(c));
  // header and base voxels
  std::vector<uint32_t> out = {kMagic, (uint32_t)B, (uint32_t)b0, (uint32_t)stages, (uint32_t)nstreams,
                               (uint32_t)n0};
  {
    const int32_t* xyz = reinterpret_cast<const int32_t*>(static_cast<char*>(c->fc_aux_host) + xyz_off);
    const uint8_t* code = reinterpret_cast<const uint8_t*>(static_cast<char*>(c->fc_aux_host) + code_off);
    BitWriter bw{out};
    for (int64_t i = 0; i < n0; ++i) {
      for (int a = 0; a < 3; ++a) bw.put((uint32_t)xyz[3 * i + a], b0);
      bw.put(code[i], 8);
    }
    bw.flush();
  }
  // every model scale and stage as interleaved streams
  const uint16_t* iv = static_cast<const uint16_t*>(c->fc_tab_host);
  std::vector<uint32_t> words;
  std::vector<int64_t> wc(nstreams);
  int64_t off = 0;
  for (int b = b0 + 1; b < B; ++b) {
    const int64_t nb = counts[b];
    for (int s = 0; s < stages; ++s) {
      words.resize((size_t)nb + 16 * (size_t)nstreams);
      const reno_status st = reno_rans_encode_streams(iv + off * per + 2 * s, nb, per, nstreams, 0, words.data(),
                                                      (int64_t)words.size(), wc.data());
      if (st != RENO_OK) return frame_fail(c, st, "rANS encode of a scale failed");
      int64_t tot = 0;
      for (int j = 0; j < nstreams; ++j) {
        out.push_back((uint32_t)wc[j]);
        tot += wc[j];
      }
      out.insert(out.end(), words.begin(), words.begin() + tot);
    }
    off += nb;
  }
  *nwords_host = (int64_t)out.size();
  if ((int64_t)out.size() > cap_words) return frame_fail(c, RENO_E_CAPACITY, "bitstream exceeds cap_words");
  std::copy(out.begin(), out.end(), out_host);
  return RENO_OK;
}

reno_status reno_decode_frame(reno_ctx* c, const uint32_t* in_host, int64_t nwords) {
  using namespace reno;
  if (!c) return RENO_E_INVALID;
  if (!in_host || nwords < kHeader) return frame_fail(c, RENO_E_INPUT, "bitstream shorter than its header");
  if (!c->have_weights) return frame_fail(c, RENO_E_STATE, "no weights set");
  const bool two = c->p.head_mode == RENO_HEAD_TWO_STAGE;
  const int stages = two ? 2 : 1, k = two ? 16 : 256;
  const int64_t B = in_host[1], b0 = in_host[2], S = in_host[4], n0 = in_host[5];
  if (in_host[0] != kMagic) return frame_fail(c, RENO_E_INPUT, "not a frame bitstream");
  if (b0 != c->b0()) return frame_fail(c, RENO_E_INPUT, "min_bit_depth differs from the context's");
  if (B <= b0 || B > c->p.max_bit_depth) return frame_fail(c, RENO_E_INPUT, "bit depth out of range");
  if ((int64_t)in_host[3] != stages) return frame_fail(c, RENO_E_INPUT, "head stages differ from the context's");
  if (S < 1 || S > RENO_RANS_MAX_STREAMS) return frame_fail(c, RENO_E_INPUT, "stream count out of range");
  if (3 * b0 + 8 > 32) return frame_fail(c, RENO_E_INVALID, "frame coding needs min_bit_depth <= 8");
  if (n0 > c->cap_pts || n0 > (int64_t(1) << (3 * b0))) return frame_fail(c, RENO_E_INPUT, "base count out of range");
  // base voxels
  FRAME_HIP(c, grow(&c->fc_aux_dev, &c->fc_aux_host, &c->fc_aux_bytes,
                    (sizeof(int32_t) * 3 + 2) * (size_t)std::max<int64_t>(c->cap_pts, 1)));
  int32_t* xyz_host = static_cast<int32_t*>(c->fc_aux_host);
  uint8_t* code_host = reinterpret_cast<uint8_t*>(xyz_host + 3 * c->cap_pts);
  uint8_t* s1_host = code_host + c->cap_pts;
  int32_t* xyz_dev = static_cast<int32_t*>(c->fc_aux_dev);
  uint8_t* code_dev = reinterpret_cast<uint8_t*>(xyz_dev + 3 * c->cap_pts);
  uint8_t* s1_dev = code_dev + c->cap_pts;
  int64_t pos = kHeader;
  {
    BitReader br{in_host + kHeader, nwords - kHeader};
    for (int64_t i = 0; i < n0; ++i) {
      uint32_t v[4];
      for (int a = 0; a < 3; ++a)
        if (!br.get((int)b0, &v[a])) return frame_fail(c, RENO_E_INPUT, "bitstream ends inside the base voxels");
      if (!br.get(8, &v[3])) return frame_fail(c, RENO_E_INPUT, "bitstream ends inside the base voxels");
      for (int a = 0; a < 3; ++a) xyz_host[3 * i + a] = (int32_t)v[a];
      code_host[i] = (uint8_t)v[3];
      if (v[3] == 0) return frame_fail(c, RENO_E_INPUT, "a base occupancy code is zero");
    }
    pos += br.pos;
  }
  if (n0 > 0) {
    FRAME_HIP(c, hipMemcpyAsync(xyz_dev, xyz_host, sizeof(int32_t) * 3 * (size_t)n0, hipMemcpyHostToDevice,
                                c->stream));
    FRAME_HIP(c, hipMemcpyAsync(code_dev, code_host, (size_t)n0, hipMemcpyHostToDevice, c->stream));
  }
  FRAME_OK(reno_set_base(c, (int)B, xyz_dev, code_dev, n0));
  // the scales: N_b follows from the codes of scale b - 1 (their popcounts),
  // so the host knows every size without asking the device
  int64_t nb = 0;
  for (int64_t i = 0; i < n0; ++i) nb += __builtin_popcount(code_host[i]);
  const uint8_t* prev = nullptr;  // codes of the scale below, on the device (base: recorded by set_base)
  std::vector<int64_t> wc(S);
  int64_t rows = 0;  // model rows so far
  for (int b = (int)b0 + 1; b < B; ++b) {
    if (nb > c->cap_pts || rows + nb > c->cap_model)
      return frame_fail(c, RENO_E_CAPACITY, "a scale exceeds the context capacity");
    rows += nb;
    FRAME_OK(reno_expand(c, b - 1, prev));
    FRAME_OK(reno_predict_probs(c, b, nullptr, nullptr));
    FRAME_HIP(c, grow(&c->fc_tab_dev, &c->fc_tab_host, &c->fc_tab_bytes,
                      sizeof(uint16_t) * (size_t)std::max<int64_t>(nb, 1) * k));
    uint16_t* tab_dev = static_cast<uint16_t*>(c->fc_tab_dev);
    const uint16_t* tab_host = static_cast<const uint16_t*>(c->fc_tab_host);
    for (int s = 0; s < stages; ++s) {
      const int stage = two ? s + 1 : 0;
      if (s == 1) {
        FRAME_HIP(c, hipMemcpyAsync(s1_dev, s1_host, (size_t)nb, hipMemcpyHostToDevice, c->stream));
        FRAME_OK(reno_predict_second(c, b, s1_dev, nullptr));
      }
      FRAME_OK(reno_symbol_cdf(c, b, stage, tab_dev));
      if (nb > 0)
        FRAME_HIP(c, hipMemcpyAsync(const_cast<uint16_t*>(tab_host), tab_dev, sizeof(uint16_t) * (size_t)nb * k,
                                    hipMemcpyDeviceToHost, c->stream));
      FRAME_HIP(c, hipStreamSynchronize(c->stream));
      if (pos + S > nwords) return frame_fail(c, RENO_E_INPUT, "bitstream ends before a scale's streams");
      int64_t tot = 0;
      for (int64_t j = 0; j < S; ++j) tot += (wc[j] = in_host[pos + j]);
      pos += S;
      if (pos + tot > nwords) return frame_fail(c, RENO_E_INPUT, "bitstream ends inside a scale's streams");
      uint8_t* sym = (two && s == 0) ? s1_host : code_host;
      const reno_status st =
          reno_rans_decode_streams(in_host + pos, wc.data(), (int)S, 0, tab_host, k, nb, sym);
      if (st != RENO_OK) {
        const reno_status dev = reno_sync(c);  // a device error explains it better
        return dev != RENO_OK ? dev : frame_fail(c, st, "rANS decode of a scale failed");
      }
      pos += tot;
    }
    int64_t nn = 0;
    for (int64_t i = 0; i < nb; ++i) {
      if (two) code_host[i] = (uint8_t)(s1_host[i] | (code_host[i] << 4));
      nn += __builtin_popcount(code_host[i]);
    }
    if (std::find(code_host, code_host + nb, uint8_t(0)) != code_host + nb)
      return frame_fail(c, RENO_E_INPUT, "a decoded occupancy code is zero");
    if (nb > 0) FRAME_HIP(c, hipMemcpyAsync(code_dev, code_host, (size_t)nb, hipMemcpyHostToDevice, c->stream));
    prev = code_dev;
    nb = nn;
  }
  if (pos != nwords) return frame_fail(c, RENO_E_INPUT, "bitstream longer than the frame");
  if (nb > c->cap_pts) return frame_fail(c, RENO_E_CAPACITY, "the finest scale exceeds the context capacity");
  FRAME_OK(reno_expand(c, (int)B - 1, prev));
  return reno_sync(c);
}

}  // extern "C"
