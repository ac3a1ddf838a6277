// C ABI of the codec hot path: argument checks, call-order state, buffer
// ownership and device-error reporting.  Every compute step is a HIP kernel
// enqueued on the context stream (see the k_*.hip files).

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>

#include "ctx.h"

namespace {

using reno::Ctx;
thread_local std::string g_create_err;

reno_status fail(Ctx* c, reno_status s, const std::string& msg) {
  if (c)
    c->err = msg;
  else
    g_create_err = msg;
  return s;
}

#define RENO_HIP(c, expr)                                                                  \
  do {                                                                                     \
    hipError_t e_ = (expr);                                                                \
    if (e_ != hipSuccess)                                                                  \
      return fail((c), RENO_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_));     \
  } while (0)

size_t round256(size_t n) { return (n + 255) & ~size_t(255); }

// device allocation, tallied into *total (bytes actually requested)
template <typename T>
hipError_t dalloc(T** p, size_t count, int64_t* total) {
  const size_t bytes = round256(count * sizeof(T) + 16);
  *total += (int64_t)bytes;
  return hipMalloc(reinterpret_cast<void**>(p), bytes);
}

bool has(uint32_t mask, int b) { return b >= 0 && b < 32 && ((mask >> b) & 1u); }
uint32_t bits_range(int lo, int hi) {  // bits lo..hi inclusive
  uint32_t m = 0;
  for (int b = lo; b <= hi; ++b) m |= 1u << b;
  return m;
}

void free_all(Ctx* c) {
  void* ptrs[] = {c->keys_a,  c->keys_b,    c->lv_key,   c->lv_code,  c->lv_parent, c->lv_fc,
                  c->lv_feat, c->d_count,   c->d_moff,   c->d_err,    c->d_hist,    c->d_ticket,
                  c->d_status, c->d_hash,   c->d_hreg,   c->h_a,      c->h_b,      c->d_nbr,     c->d_lse,
                  c->d_partial, c->d_total, c->w_head,   c->w_hbias,  c->w_head_plain,
                  c->d_lse2,    c->w_emb,   c->d_s1,     c->w_head_t, c->d_perm,
                  c->h_c,       c->h_d,     c->w_embo,   c->w_embd};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  for (int l = 0; l < RENO_MAX_LAYERS; ++l) {
    if (c->w_conv[l]) (void)hipFree(c->w_conv[l]);
    if (c->w_bias[l]) (void)hipFree(c->w_bias[l]);
  }
  if (c->h_total) (void)hipHostFree(c->h_total);
  if (c->h_count) (void)hipHostFree(c->h_count);
  if (c->h_err) (void)hipHostFree(c->h_err);
  for (hipEvent_t ev : c->prof_pool) (void)hipEventDestroy(ev);
  c->prof_pool.clear();
  reno::frame_free(*c);
}

// Waits for the stream and turns latched device errors into a status.
reno_status sync_check(Ctx* c) {
  RENO_HIP(c, hipMemcpyAsync(c->h_err, c->d_err, sizeof(uint32_t), hipMemcpyDeviceToHost, c->stream));
  RENO_HIP(c, hipStreamSynchronize(c->stream));
  const uint32_t e = *c->h_err;
  if (e == 0) return RENO_OK;
  std::string msg = "device reported:";
  if (e & reno::ERR_NONFINITE) msg += " non-finite input coordinate;";
  if (e & reno::ERR_ZERO_CODE) msg += " zero occupancy code;";
  if (e & reno::ERR_BASE_ORDER) msg += " base voxels not strictly ascending in Morton order;";
  if (e & reno::ERR_BASE_RANGE) msg += " base voxel outside the base grid;";
  if (e & reno::ERR_CAPACITY) msg += " frame exceeds the context capacity;";
  if (e & reno::ERR_HASH_FULL) msg += " coordinate hash full;";
  if (e & reno::ERR_SPIN) msg += " internal: look-back wait bound exceeded;";
  if (e & reno::ERR_DUP_KEY) msg += " internal: duplicate hash key;";
  if (e & reno::ERR_INTERNAL) msg += " internal: consistency check failed;";
  if (e & reno::ERR_SYMBOL) msg += " first sub-code outside 0..15;";
  if (e & reno::ERR_FRAMES) msg += " frame ranges or frame ids of the batch malformed;";
  if (e & reno::ERR_STREAM) msg += " entropy-coded stream of the bitstream malformed;";
  // a malformed bitstream explains what follows from decoding it (codes of
  // zero, scales past the capacity)
  if (e & reno::ERR_STREAM) return fail(c, RENO_E_INPUT, msg);
  if (e & (reno::ERR_CAPACITY | reno::ERR_HASH_FULL)) return fail(c, RENO_E_CAPACITY, msg);
  if (e & (reno::ERR_SPIN | reno::ERR_DUP_KEY | reno::ERR_INTERNAL)) return fail(c, RENO_E_HIP, msg);
  return fail(c, RENO_E_INPUT, msg);
}

// Zeroes the per-frame counters, tickets, look-back state and hash.
reno_status frame_init(Ctx* c) {
  void* p[8];
  size_t n[8];
  const int k = reno::frame_clear(*c, p, n);
  RENO_HIP(c, reno::launch_zero(*c, p, n, k));
  return RENO_OK;
}

// frame-id bits of a batch: ceil(log2(frames))
int frame_bits(int frames) {
  int fb = 0;
  while ((1 << fb) < frames) ++fb;
  return fb;
}

bool model_scale(const Ctx* c, int b) { return c->B > 0 && b > c->b0() && b < c->B; }
// the two-stage head needs stage 2 of a scale before its code lengths
bool stage2_ok(const Ctx* c, int b) {
  return c->p.head_mode != RENO_HEAD_TWO_STAGE || has(c->have_pred2, b);
}

}  // namespace

extern "C" {

const char* reno_last_error(const reno_ctx* ctx) {
  return ctx ? ctx->err.c_str() : g_create_err.c_str();
}

reno_status reno_create(const reno_params* p, void* hip_stream, reno_ctx** out) {
  if (!p || !out) return fail(nullptr, RENO_E_INVALID, "null argument");
  *out = nullptr;
  if (p->max_points < 1 || p->max_points >= (int64_t(1) << 30))
    return fail(nullptr, RENO_E_INVALID, "max_points must be in [1, 2^30)");
  if (p->max_bit_depth < 1 || p->max_bit_depth > RENO_MAX_BIT_DEPTH)
    return fail(nullptr, RENO_E_INVALID, "max_bit_depth must be in [1, 21]");
  if (p->min_bit_depth < 0 || p->min_bit_depth >= p->max_bit_depth)
    return fail(nullptr, RENO_E_INVALID, "min_bit_depth must be in [0, max_bit_depth)");
  if (!(p->range_m > 0.0) || !std::isfinite(p->range_m))
    return fail(nullptr, RENO_E_INVALID, "range_m must be positive and finite");
  if (p->in_features != RENO_IN_FEATURES)
    return fail(nullptr, RENO_E_INVALID, "in_features must be 11");
  const bool top_mode = p->model_mode == RENO_MODEL_TOP;
  if (!(p->channels == 16 || p->channels == 32 || (top_mode && (p->channels == 64 || p->channels == 128))))
    return fail(nullptr, RENO_E_INVALID, "channels must be 16 or 32 (full predictor: 16, 32, 64 or 128)");
  if (p->kernel_size != 0 && p->kernel_size != 3 && !(top_mode && p->kernel_size == 5))
    return fail(nullptr, RENO_E_INVALID, "kernel_size must be 3 (full predictor: 3 or 5)");
  if (p->layers < 1 || p->layers > RENO_MAX_LAYERS)
    return fail(nullptr, RENO_E_INVALID, "layers must be in [1, 8]");
  if (p->head_mode != RENO_HEAD_ONE_STAGE && p->head_mode != RENO_HEAD_TWO_STAGE)
    return fail(nullptr, RENO_E_INVALID, "head_mode must be RENO_HEAD_ONE_STAGE or RENO_HEAD_TWO_STAGE");
  if (p->precision != RENO_PREC_FP32 && p->precision != RENO_PREC_BF16X3)
    return fail(nullptr, RENO_E_INVALID, "precision must be RENO_PREC_FP32 or RENO_PREC_BF16X3");
  if (p->model_mode != RENO_MODEL_PLAIN && p->model_mode != RENO_MODEL_TOP)
    return fail(nullptr, RENO_E_INVALID, "model_mode must be RENO_MODEL_PLAIN or RENO_MODEL_TOP");
  if (p->model_mode == RENO_MODEL_TOP && p->precision != RENO_PREC_FP32)
    return fail(nullptr, RENO_E_INVALID, "the full predictor runs in RENO_PREC_FP32 only");
  // N_b <= N_{b+1} <= max_points, so (model scales) x max_points always suffices
  const int64_t nmodel = p->max_bit_depth - p->min_bit_depth - 1 > 0
                             ? p->max_bit_depth - p->min_bit_depth - 1 : 1;
  int64_t cap_model = p->max_model_voxels > 0 ? p->max_model_voxels : nmodel * p->max_points;
  if (cap_model >= (int64_t(1) << 30))
    return fail(nullptr, RENO_E_INVALID, "max_model_voxels must be below 2^30");

  reno_ctx* c = new reno_ctx();
  c->p = *p;
  c->p.max_model_voxels = cap_model;
  c->stream = static_cast<hipStream_t>(hip_stream);
  if (hipGetDevice(&c->device) != hipSuccess) {
    delete c;
    return fail(nullptr, RENO_E_HIP, "no HIP device");
  }
  c->cap_pts = p->max_points;
  c->cap_model = cap_model;
  c->nlv = p->max_bit_depth - p->min_bit_depth + 1;
  int lg = 10;
  while ((int64_t(1) << lg) * 3 < cap_model * 4 && lg < 31) ++lg;  // load factor <= 3/4
  c->hash_lg = lg;
  c->sort_tiles = (c->cap_pts + reno::SORT_TILE - 1) / reno::SORT_TILE;
  c->pyr_tiles = (c->cap_pts + reno::PYR_TILE - 1) / reno::PYR_TILE;
  c->exp_tiles = (c->cap_pts + reno::EXP_TILE - 1) / reno::EXP_TILE;
  c->status_words = (int64_t)reno::MAX_PASSES * c->sort_tiles * reno::RADIX +
                    c->pyr_tiles * reno::NLEV + (int64_t)reno::NLEV * c->exp_tiles;
  const int C = p->channels;
  const size_t lvn = (size_t)c->nlv * c->cap_pts;
  hipError_t e = hipSuccess;
  auto A = [&](hipError_t r) {
    if (e == hipSuccess) e = r;
  };
  A(dalloc(&c->keys_a, c->cap_pts, &c->device_bytes));
  A(dalloc(&c->keys_b, c->cap_pts, &c->device_bytes));
  A(dalloc(&c->lv_key, lvn, &c->device_bytes));
  A(dalloc(&c->lv_code, lvn, &c->device_bytes));
  A(dalloc(&c->lv_parent, lvn, &c->device_bytes));
  A(dalloc(&c->lv_fc, lvn, &c->device_bytes));
  A(dalloc(&c->lv_feat, lvn + 8, &c->device_bytes));  // entry lvn stays zero: absent-neighbour input
  A(dalloc(&c->d_count, reno::NLEV, &c->device_bytes));
  A(dalloc(&c->d_moff, reno::NLEV + 1, &c->device_bytes));
  A(dalloc(&c->d_err, 4, &c->device_bytes));
  A(dalloc(&c->d_hist, reno::MAX_PASSES * reno::RADIX, &c->device_bytes));
  A(dalloc(&c->d_ticket, reno::TICKETS, &c->device_bytes));
  A(dalloc(&c->d_status, (size_t)c->status_words, &c->device_bytes));
  A(dalloc(&c->d_hash, size_t(1) << c->hash_lg, &c->device_bytes));
  A(dalloc(&c->d_hreg, (size_t)RENO_MAX_FRAMES + 1, &c->device_bytes));
  const bool top = c->top();
  const size_t rows = (size_t)c->cap_rows();  // row cap_model stays zero
  A(dalloc(&c->h_a, rows * C, &c->device_bytes));
  A(dalloc(&c->h_b, rows * C, &c->device_bytes));
  if (top) {
    A(dalloc(&c->h_c, rows * C, &c->device_bytes));
    A(dalloc(&c->h_d, rows * C, &c->device_bytes));
    A(dalloc(&c->w_embo, (size_t)256 * C, &c->device_bytes));
    A(dalloc(&c->w_embd, (size_t)8 * C, &c->device_bytes));
  }
  A(dalloc(&c->d_nbr, rows * c->nbr_stride(), &c->device_bytes));
  A(dalloc(&c->d_lse, (size_t)cap_model, &c->device_bytes));
  A(dalloc(&c->d_lse2, (size_t)cap_model, &c->device_bytes));
  A(dalloc(&c->d_perm, rows, &c->device_bytes));
  A(dalloc(&c->d_s1, (size_t)cap_model, &c->device_bytes));
  A(dalloc(&c->d_partial, (size_t)reno::NLEV * ((c->cap_pts + 63) / 64), &c->device_bytes));
  A(dalloc(&c->d_total, reno::NLEV, &c->device_bytes));
  int c_in = top ? C : RENO_IN_FEATURES;
  for (int l = 0; l < (top ? 4 : p->layers); ++l) {
    const int KS = (c_in + 3) / 4, KSP = (KS + 3) & ~3;
    // fp32: KSP floats per (offset, column block, lane); bf16x3: 8 words
    A(dalloc(&c->w_conv[l], (size_t)(top ? c->kvol() : 27) * (C / 16) * 64 * std::max(KSP, 8),
             &c->device_bytes));
    A(dalloc(&c->w_bias[l], (size_t)C, &c->device_bytes));
    c_in = C;
  }
  A(dalloc(&c->w_head, (size_t)16 * 64 * std::max(C / 4, 8), &c->device_bytes));
  A(dalloc(&c->w_hbias, 256, &c->device_bytes));
  A(dalloc(&c->w_head_plain, (size_t)C * 256, &c->device_bytes));
  A(dalloc(&c->w_emb, (size_t)16 * C, &c->device_bytes));
  A(dalloc(&c->w_head_t, (size_t)256 * C, &c->device_bytes));
  A(hipHostMalloc(reinterpret_cast<void**>(&c->h_total), sizeof(double) * reno::NLEV, 0));
  A(hipHostMalloc(reinterpret_cast<void**>(&c->h_count), sizeof(int32_t) * reno::NLEV, 0));
  A(hipHostMalloc(reinterpret_cast<void**>(&c->h_err), 64, 0));
  if (e != hipSuccess) {
    const std::string msg = std::string("allocation failed: ") + hipGetErrorString(e);
    free_all(c);
    delete c;
    return fail(nullptr, e == hipErrorOutOfMemory ? RENO_E_NOMEM : RENO_E_HIP, msg);
  }
  // tickets start at zero (every frame clears them again); the reserved zero
  // row of each feature buffer and the zero input-bit entry are never written
  // afterwards
  e = hipMemsetAsync(c->d_ticket, 0, sizeof(uint32_t) * reno::TICKETS, c->stream);
  if (e == hipSuccess)
    e = hipMemsetAsync(c->h_a + (size_t)cap_model * C, 0, sizeof(float) * C, c->stream);
  if (e == hipSuccess)
    e = hipMemsetAsync(c->h_b + (size_t)cap_model * C, 0, sizeof(float) * C, c->stream);
  if (e == hipSuccess && top)
    e = hipMemsetAsync(c->h_c + (size_t)cap_model * C, 0, sizeof(float) * C, c->stream);
  if (e == hipSuccess && top)
    e = hipMemsetAsync(c->h_d + (size_t)cap_model * C, 0, sizeof(float) * C, c->stream);
  if (e == hipSuccess) e = hipMemsetAsync(c->lv_feat + lvn, 0, 16, c->stream);
  if (e == hipSuccess) e = hipStreamSynchronize(c->stream);
  if (e != hipSuccess) {
    const std::string msg = std::string("init failed: ") + hipGetErrorString(e);
    free_all(c);
    delete c;
    return fail(nullptr, RENO_E_HIP, msg);
  }
  *out = c;
  return RENO_OK;
}

reno_status reno_destroy(reno_ctx* c) {
  if (!c) return RENO_E_INVALID;
  (void)hipStreamSynchronize(c->stream);
  free_all(c);
  delete c;
  return RENO_OK;
}

reno_status reno_memory_info(const reno_ctx* c, int64_t* info_host) {
  if (!c || !info_host) return RENO_E_INVALID;
  info_host[0] = int64_t(1) << c->hash_lg;
  info_host[1] = c->status_words;
  info_host[2] = c->cap_model;
  info_host[3] = c->device_bytes;
  return RENO_OK;
}

reno_status reno_sync(reno_ctx* c) {
  if (!c) return RENO_E_INVALID;
  return sync_check(c);
}

reno_status reno_set_weights(reno_ctx* c, const reno_weights* w) {
  if (!c || !w) return fail(c, RENO_E_INVALID, "null argument");
  if (c->top()) {
    for (int l = 0; l < 4; ++l)
      if (!w->top_w[l] || !w->top_b[l]) return fail(c, RENO_E_INVALID, "missing residual-block weights");
    if (!w->emb_o || !w->emb_d) return fail(c, RENO_E_INVALID, "missing embedding weights");
  } else {
    for (int l = 0; l < c->p.layers; ++l)
      if (!w->conv_w[l] || !w->conv_b[l]) return fail(c, RENO_E_INVALID, "missing conv weights");
  }
  if (c->p.head_mode == RENO_HEAD_TWO_STAGE) {
    if (!w->head1_w || !w->head1_b || !w->emb_s1 || !w->head2_w || !w->head2_b)
      return fail(c, RENO_E_INVALID, "missing two-stage head weights");
  } else if (!w->head_w || !w->head_b) {
    return fail(c, RENO_E_INVALID, "missing head weights");
  }
  RENO_HIP(c, reno::launch_pack_weights(*c, *w));
  c->have_weights = true;
  return RENO_OK;
}

reno_status reno_build_pyramid(reno_ctx* c, const float* points, int64_t n, int bit_depth) {
  return reno_build_pyramid_frames(c, points, n, nullptr, 1, bit_depth);
}

reno_status reno_build_pyramid_frames(reno_ctx* c, const float* points, int64_t n, const int64_t* frame_start,
                                      int frames, int bit_depth) {
  if (!c) return RENO_E_INVALID;
  if (n < 0 || n > c->cap_pts) return fail(c, RENO_E_INVALID, "point count out of range");
  if (n > 0 && !points) return fail(c, RENO_E_INVALID, "null points");
  if (bit_depth <= c->b0() || bit_depth > c->p.max_bit_depth)
    return fail(c, RENO_E_INVALID, "bit_depth must be in (min_bit_depth, max_bit_depth]");
  if (frames < 1 || frames > RENO_MAX_FRAMES) return fail(c, RENO_E_INVALID, "frames must be in [1, 1024]");
  if (frames > 1 && !frame_start) return fail(c, RENO_E_INVALID, "null frame_start");
  const int fb = frame_bits(frames);
  if (3 * bit_depth + fb > 63) return fail(c, RENO_E_INVALID, "3 * bit_depth + frame-id bits exceed 63");
  const int B = bit_depth;
  c->B = B;
  c->encoder = true;
  c->npoints = n;
  c->frames = frames;
  c->fbits = fb;
  c->have_level = bits_range(c->b0(), B);
  c->have_codes = bits_range(c->b0(), B - 1);
  c->have_pred = 0;
  c->have_pred2 = 0;
  reno_status s = frame_init(c);
  if (s != RENO_OK) return s;
  if (n == 0) return RENO_OK;
  const int passes = (3 * B + fb + reno::RADIX_BITS - 1) / reno::RADIX_BITS;
  RENO_HIP(c, reno::launch_quantize(*c, points, n, B, passes, frames > 1 ? frame_start : nullptr, frames));
  uint64_t* src = c->keys_a;
  uint64_t* dst = c->keys_b;
  for (int ps = 0; ps < passes; ++ps) {
    RENO_HIP(c, reno::launch_sort_pass(*c, src, dst, n, ps));
    uint64_t* t = src;
    src = dst;
    dst = t;
  }
  RENO_HIP(c, reno::launch_pyramid(*c, src, n, B));
  RENO_HIP(c, reno::launch_codes(*c, B));
  return RENO_OK;
}

reno_status reno_set_base(reno_ctx* c, int bit_depth, const int32_t* xyz, const uint8_t* codes,
                          int64_t n) {
  return reno_set_base_frames(c, bit_depth, xyz, nullptr, codes, n, 1);
}

reno_status reno_set_base_frames(reno_ctx* c, int bit_depth, const int32_t* xyz, const int32_t* frame_of,
                                 const uint8_t* codes, int64_t n, int frames) {
  if (!c) return RENO_E_INVALID;
  if (bit_depth <= c->b0() || bit_depth > c->p.max_bit_depth)
    return fail(c, RENO_E_INVALID, "bit_depth must be in (min_bit_depth, max_bit_depth]");
  if (frames < 1 || frames > RENO_MAX_FRAMES) return fail(c, RENO_E_INVALID, "frames must be in [1, 1024]");
  if (frames > 1 && n > 0 && !frame_of) return fail(c, RENO_E_INVALID, "null frame ids");
  const int fb = frame_bits(frames);
  if (3 * bit_depth + fb > 63) return fail(c, RENO_E_INVALID, "3 * bit_depth + frame-id bits exceed 63");
  const int64_t grid = int64_t(1) << (3 * c->b0());
  if (n < 0 || n > c->cap_pts || n > grid * frames) return fail(c, RENO_E_INVALID, "base count out of range");
  if (n > 0 && (!xyz || !codes)) return fail(c, RENO_E_INVALID, "null base arrays");
  c->B = bit_depth;
  c->encoder = false;
  c->npoints = 0;
  c->frames = frames;
  c->fbits = fb;
  c->have_level = 1u << c->b0();
  c->have_codes = 1u << c->b0();
  c->have_pred = 0;
  c->have_pred2 = 0;
  if (reno::clear_set_base_fits(n)) {  // a small base scale: the clear and the base scale in one launch
    RENO_HIP(c, reno::launch_clear_set_base(*c, xyz, frames > 1 ? frame_of : nullptr, codes, n));
    return RENO_OK;
  }
  reno_status s = frame_init(c);
  if (s != RENO_OK) return s;
  RENO_HIP(c, reno::launch_set_base(*c, xyz, frames > 1 ? frame_of : nullptr, codes, n, bit_depth));
  return RENO_OK;
}

reno_status reno_expand(reno_ctx* c, int scale, const uint8_t* codes) {
  if (!c) return RENO_E_INVALID;
  if (c->B == 0) return fail(c, RENO_E_STATE, "no frame");
  if (scale < c->b0() || scale >= c->B) return fail(c, RENO_E_INVALID, "scale out of range");
  if (!has(c->have_level, scale)) return fail(c, RENO_E_STATE, "scale not built yet");
  if (has(c->have_level, scale + 1))
    return fail(c, RENO_E_STATE, "the next scale already exists in this frame");
  if (!codes && !has(c->have_codes, scale)) return fail(c, RENO_E_STATE, "codes of the scale unknown");
  RENO_HIP(c, reno::launch_expand(*c, scale, codes, c->B));
  c->have_codes |= 1u << scale;
  c->have_level |= 1u << (scale + 1);
  return RENO_OK;
}

reno_status reno_expand_noalloc(const uint64_t* keys, const uint8_t* codes, int64_t n,
                                uint64_t* child_keys, int32_t* child_parent, int64_t cap_children,
                                int32_t* first_child, int64_t* result, void* hip_stream) {
  if (n < 0 || n > RENO_NOALLOC_MAX_PARENTS)
    return fail(nullptr, RENO_E_INVALID, "n must be in [0, RENO_NOALLOC_MAX_PARENTS]");
  if (cap_children < 0 || cap_children >= (int64_t(1) << 31))
    return fail(nullptr, RENO_E_INVALID, "cap_children must be in [0, 2^31)");
  if (!result) return fail(nullptr, RENO_E_INVALID, "null result");
  if (n > 0 && (!keys || !codes)) return fail(nullptr, RENO_E_INVALID, "null input");
  if (cap_children > 0 && (!child_keys || !child_parent)) return fail(nullptr, RENO_E_INVALID, "null output");
  RENO_HIP(nullptr, reno::launch_expand_noalloc(keys, codes, n, child_keys, child_parent, cap_children,
                                                first_child, result, static_cast<hipStream_t>(hip_stream)));
  return RENO_OK;
}

reno_status reno_scale_counts(reno_ctx* c, int64_t* counts_host) {
  if (!c || !counts_host) return fail(c, RENO_E_INVALID, "null argument");
  RENO_HIP(c, hipMemcpyAsync(c->h_count, c->d_count, sizeof(int32_t) * reno::NLEV,
                             hipMemcpyDeviceToHost, c->stream));
  reno_status s = sync_check(c);
  if (s != RENO_OK) return s;
  for (int b = 0; b < reno::NLEV; ++b)
    counts_host[b] = (c->B > 0 && has(c->have_level, b)) ? (int64_t)c->h_count[b] : 0;
  return RENO_OK;
}

reno_status reno_num_voxels(reno_ctx* c, int scale, int64_t* n_host) {
  if (!c || !n_host) return fail(c, RENO_E_INVALID, "null argument");
  if (!has(c->have_level, scale)) return fail(c, RENO_E_STATE, "scale not built");
  RENO_HIP(c, hipMemcpyAsync(c->h_count, c->d_count, sizeof(int32_t) * reno::NLEV,
                             hipMemcpyDeviceToHost, c->stream));
  reno_status s = sync_check(c);
  if (s != RENO_OK) return s;
  *n_host = c->h_count[scale];
  return RENO_OK;
}

reno_status reno_coords(reno_ctx* c, int scale, int32_t* xyz, uint64_t* keys) {
  if (!c) return RENO_E_INVALID;
  if (!has(c->have_level, scale)) return fail(c, RENO_E_STATE, "scale not built");
  if (!xyz && !keys) return RENO_OK;
  RENO_HIP(c, reno::launch_coords(*c, scale, xyz, keys));
  return RENO_OK;
}

reno_status reno_occupancy_codes(reno_ctx* c, int scale, uint8_t* codes) {
  if (!c || !codes) return fail(c, RENO_E_INVALID, "null argument");
  if (!has(c->have_codes, scale)) return fail(c, RENO_E_STATE, "codes of the scale unknown");
  RENO_HIP(c, reno::launch_copy_level_u8(*c, scale, codes));
  return RENO_OK;
}

reno_status reno_parent_rows(reno_ctx* c, int scale, int32_t* parent) {
  if (!c || !parent) return fail(c, RENO_E_INVALID, "null argument");
  if (!has(c->have_level, scale)) return fail(c, RENO_E_STATE, "scale not built");
  RENO_HIP(c, reno::launch_copy_level_i32(*c, scale, c->lv_parent + c->lv(scale), parent));
  return RENO_OK;
}

reno_status reno_predict_probs(reno_ctx* c, int scale, const reno_weights* weights, float* logits) {
  if (!c) return RENO_E_INVALID;
  if (c->B == 0) return fail(c, RENO_E_STATE, "no frame");
  if (weights) {
    reno_status s = reno_set_weights(c, weights);
    if (s != RENO_OK) return s;
  }
  if (!c->have_weights) return fail(c, RENO_E_STATE, "no weights set");
  int lo, hi;
  if (scale == RENO_ALL_SCALES) {
    lo = c->b0() + 1;
    hi = c->B - 1;
    if (lo > hi) return RENO_OK;
    for (int b = lo; b <= hi; ++b)
      if (!has(c->have_level, b) || !has(c->have_codes, b - 1))
        return fail(c, RENO_E_STATE, "every model scale and its parent codes must exist");
  } else {
    if (!model_scale(c, scale)) return fail(c, RENO_E_INVALID, "not a model scale");
    if (!has(c->have_level, scale) || !has(c->have_codes, scale - 1))
      return fail(c, RENO_E_STATE, "scale or the codes of its parent scale unknown");
    lo = hi = scale;
  }
  const bool two = c->p.head_mode == RENO_HEAD_TWO_STAGE;
  const bool second = two && (c->have_codes & bits_range(lo, hi)) == bits_range(lo, hi);
  RENO_HIP(c, reno::launch_model(*c, lo, hi, logits, second));
  c->have_pred |= bits_range(lo, hi);
  c->have_pred2 &= ~bits_range(lo, hi);
  if (second) c->have_pred2 |= bits_range(lo, hi);
  return RENO_OK;
}

reno_status reno_predict_second(reno_ctx* c, int scale, const uint8_t* s1, float* logits2) {
  if (!c) return RENO_E_INVALID;
  if (c->p.head_mode != RENO_HEAD_TWO_STAGE) return fail(c, RENO_E_STATE, "one-stage context");
  if (c->B == 0) return fail(c, RENO_E_STATE, "no frame");
  if (!model_scale(c, scale)) return fail(c, RENO_E_INVALID, "not a model scale");
  if (!has(c->have_pred, scale)) return fail(c, RENO_E_STATE, "predict_probs of the scale not run");
  if (!s1 && !has(c->have_codes, scale))
    return fail(c, RENO_E_STATE, "no first sub-codes given and the codes of the scale unknown");
  RENO_HIP(c, reno::launch_head2(*c, scale, s1, logits2));
  c->have_pred2 |= 1u << scale;
  return RENO_OK;
}

reno_status reno_code_length(reno_ctx* c, int scale, float* bits_per_voxel, double* total_host) {
  if (!c) return RENO_E_INVALID;
  if (c->B == 0) return fail(c, RENO_E_STATE, "no frame");
  const int b0 = c->b0();
  double base_bits = 0.0;
  bool with_base = false;
  int lo = 0, hi = -1;
  if (scale == RENO_ALL_SCALES) {
    with_base = true;
    lo = b0 + 1;
    hi = c->B - 1;
    for (int b = lo; b <= hi; ++b)
      if (!has(c->have_pred, b) || !has(c->have_codes, b) || !stage2_ok(c, b))
        return fail(c, RENO_E_STATE, "every model scale needs predict_probs and its codes");
  } else if (scale == b0) {
    if (bits_per_voxel) return fail(c, RENO_E_INVALID, "the base scale has no per-voxel bits");
    with_base = true;
  } else {
    if (!model_scale(c, scale)) return fail(c, RENO_E_INVALID, "not a model scale");
    if (!has(c->have_pred, scale) || !has(c->have_codes, scale) || !stage2_ok(c, scale))
      return fail(c, RENO_E_STATE, "scale needs predict_probs and its codes");
    lo = hi = scale;
  }
  if (lo <= hi) RENO_HIP(c, reno::launch_code_length(*c, lo, hi, bits_per_voxel));
  if (!total_host) return RENO_OK;
  RENO_HIP(c, hipMemcpyAsync(c->h_total, c->d_total, sizeof(double) * reno::NLEV,
                             hipMemcpyDeviceToHost, c->stream));
  RENO_HIP(c, hipMemcpyAsync(c->h_count, c->d_count, sizeof(int32_t) * reno::NLEV,
                             hipMemcpyDeviceToHost, c->stream));
  reno_status s = sync_check(c);
  if (s != RENO_OK) return s;
  if (with_base) base_bits = 32.0 * c->frames + (double)c->h_count[b0] * (3.0 * b0 + 8.0);
  double t = base_bits;
  for (int b = lo; b <= hi; ++b) t += c->h_total[b];
  *total_host = t;
  return RENO_OK;
}

reno_status reno_neighbor_map(reno_ctx* c, int scale, int32_t* map) {
  if (!c || !map) return fail(c, RENO_E_INVALID, "null argument");
  if (!has(c->have_pred, scale)) return fail(c, RENO_E_STATE, "predict_probs of the scale not run");
  RENO_HIP(c, reno::launch_neighbor_map(*c, scale, map));
  return RENO_OK;
}

reno_status reno_symbol_freqs(reno_ctx* c, int scale, uint16_t* freq) {
  if (!c || !freq) return fail(c, RENO_E_INVALID, "null argument");
  if (c->p.head_mode != RENO_HEAD_ONE_STAGE)
    return fail(c, RENO_E_STATE, "symbol tables are built for the one-stage head only");
  if (!has(c->have_pred, scale)) return fail(c, RENO_E_STATE, "predict_probs of the scale not run");
  RENO_HIP(c, reno::launch_symbol_freqs(*c, scale, freq));
  return RENO_OK;
}

reno_status reno_symbol_freqs16(reno_ctx* c, int scale, int stage, uint16_t* freq) {
  if (!c || !freq) return fail(c, RENO_E_INVALID, "null argument");
  if (c->p.head_mode != RENO_HEAD_TWO_STAGE) return fail(c, RENO_E_STATE, "one-stage context");
  if (stage != 1 && stage != 2) return fail(c, RENO_E_INVALID, "stage must be 1 or 2");
  if (!model_scale(c, scale)) return fail(c, RENO_E_INVALID, "not a model scale");
  if (!has(stage == 1 ? c->have_pred : c->have_pred2, scale))
    return fail(c, RENO_E_STATE, stage == 1 ? "predict_probs of the scale not run"
                                            : "stage 2 of the scale not run");
  RENO_HIP(c, reno::launch_symbol_freqs16(*c, scale, stage, freq));
  return RENO_OK;
}

reno_status reno_symbol_cdf(reno_ctx* c, int scale, int stage, uint16_t* start) {
  if (!c || !start) return fail(c, RENO_E_INVALID, "null argument");
  if (!model_scale(c, scale)) return fail(c, RENO_E_INVALID, "not a model scale");
  const bool two = c->p.head_mode == RENO_HEAD_TWO_STAGE;
  if (two ? (stage != 1 && stage != 2) : stage != 0)
    return fail(c, RENO_E_INVALID, two ? "stage must be 1 or 2 with the two-stage head"
                                       : "stage must be 0 with the one-stage head");
  if (!has(stage == 2 ? c->have_pred2 : c->have_pred, scale))
    return fail(c, RENO_E_STATE, stage == 2 ? "stage 2 of the scale not run" : "predict_probs of the scale not run");
  RENO_HIP(c, reno::launch_symbol_cdf(*c, scale, stage, start));
  return RENO_OK;
}

reno_status reno_symbol_intervals(reno_ctx* c, int scale, uint16_t* iv) {
  if (!c || !iv) return fail(c, RENO_E_INVALID, "null argument");
  if (c->B == 0) return fail(c, RENO_E_STATE, "no frame");
  int lo, hi;
  if (scale == RENO_ALL_SCALES) {
    lo = c->b0() + 1;
    hi = c->B - 1;
    if (lo > hi) return RENO_OK;
  } else {
    if (!model_scale(c, scale)) return fail(c, RENO_E_INVALID, "not a model scale");
    lo = hi = scale;
  }
  for (int b = lo; b <= hi; ++b)
    if (!has(c->have_pred, b) || !has(c->have_codes, b) || !stage2_ok(c, b))
      return fail(c, RENO_E_STATE, "intervals need predict_probs (both stages) and the codes");
  RENO_HIP(c, reno::launch_symbol_intervals(*c, lo, hi, iv));
  return RENO_OK;
}

reno_status reno_profile(reno_ctx* c, uint32_t kind_mask) {
  if (!c) return RENO_E_INVALID;
  if (kind_mask >> RENO_K_COUNT) return fail(c, RENO_E_INVALID, "unknown kernel kind");
  RENO_HIP(c, hipStreamSynchronize(c->stream));
  const size_t pool = 2 * 16384;
  while (kind_mask && c->prof_pool.size() < pool) {
    hipEvent_t ev;
    RENO_HIP(c, hipEventCreate(&ev));
    c->prof_pool.push_back(ev);
  }
  c->prof_mask = kind_mask;
  c->prof_used = 0;
  c->prof_recs.clear();
  return RENO_OK;
}

reno_status reno_profile_read(reno_ctx* c, double* ms_host, int64_t* launches_host) {
  if (!c || !ms_host || !launches_host) return fail(c, RENO_E_INVALID, "null argument");
  RENO_HIP(c, hipStreamSynchronize(c->stream));
  for (int k = 0; k < RENO_K_COUNT; ++k) {
    ms_host[k] = 0.0;
    launches_host[k] = 0;
  }
  for (const reno::ProfRec& r : c->prof_recs) {
    float ms = 0.0f;
    RENO_HIP(c, hipEventElapsedTime(&ms, r.a, r.b));
    ms_host[r.kind] += ms;
    launches_host[r.kind] += 1;
  }
  c->prof_used = 0;
  c->prof_recs.clear();
  return RENO_OK;
}

}  // extern "C"
