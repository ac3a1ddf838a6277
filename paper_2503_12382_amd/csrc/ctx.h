// Context of one codec stream: capacities, device buffers and the host-side
// call-order state.  Shared by the C-ABI layer (api.cpp) and the kernel
// launchers.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>
#include <string>
#include <vector>

#include "../../include/reno.h"
#include "dev.h"

namespace reno {

constexpr int NLEV = RENO_MAX_BIT_DEPTH + 1;   // bit depths 0 .. 21
constexpr int SORT_THREADS = 256;
constexpr int SORT_KPT = 4;                     // keys per thread per sort tile
constexpr int SORT_TILE = SORT_THREADS * SORT_KPT;
constexpr int SORT_KPT_BIG = 16;                // keys per thread for inputs of SORT_BIG_N keys or more
constexpr int64_t SORT_BIG_N = int64_t(1) << 22;
constexpr int RADIX_BITS = 8;
constexpr int RADIX = 1 << RADIX_BITS;
constexpr int MAX_PASSES = (3 * RENO_MAX_BIT_DEPTH + RADIX_BITS - 1) / RADIX_BITS;
constexpr int PYR_THREADS = 256;
constexpr int PYR_KPT = 4;
constexpr int PYR_TILE = PYR_THREADS * PYR_KPT;
constexpr int EXP_THREADS = 512;
constexpr int EXP_KPT = 1;                      // parents per thread: a thread's hash inserts wait for their CAS in turn
constexpr int EXP_TILE = EXP_THREADS * EXP_KPT;
constexpr int TICKETS = 64;
constexpr int NBR_STRIDE = 32;                  // neighbour-map row: 27 offsets + 5 padding

// ticket slots
constexpr int TK_SORT = 0;        // + pass
constexpr int TK_PYR = 16;
constexpr int TK_EXPAND = 17;     // + scale (decoder: one per expand call)

struct ProfRec {
  int kind;
  hipEvent_t a, b;
};

struct Ctx {
  reno_params p{};
  hipStream_t stream = nullptr;
  int device = 0;
  std::string err;

  // capacities
  int64_t cap_pts = 0;      // voxels per scale and raw points
  int64_t cap_model = 0;    // sum of model-scale voxels
  int nlv = 0;              // allocated scales: b0 .. max_bit_depth
  int hash_lg = 0;
  int64_t sort_tiles = 0;   // max tiles of one sort pass
  int64_t status_words = 0; // look-back status capacity (uint32)
  int64_t device_bytes = 0; // device memory allocated by reno_create

  // per-scale regions: scale b lives at (b - b0) * cap_pts
  uint64_t* keys_a = nullptr;   // sort ping-pong [cap_pts]
  uint64_t* keys_b = nullptr;
  uint64_t* lv_key = nullptr;   // Morton keys of V_b
  uint8_t* lv_code = nullptr;   // O_b
  int32_t* lv_parent = nullptr; // row of the parent in V_{b-1}
  int32_t* lv_fc = nullptr;     // row of the first child in V_{b+1}
  uint16_t* lv_feat = nullptr;  // delta | O_{b-1}[parent] << 3  (layer-1 input bits)

  // device scalars / small arrays
  int32_t* d_count = nullptr;   // [NLEV] N_b
  int32_t* d_moff = nullptr;    // [NLEV] first packed model row of scale b
  uint32_t* d_err = nullptr;    // [1] latched error bits
  uint32_t* d_hist = nullptr;   // [MAX_PASSES][RADIX]
  uint32_t* d_ticket = nullptr; // [TICKETS]
  uint32_t* d_status = nullptr; // look-back status words
  HashSlot* d_hash = nullptr;   // [1 << hash_lg]
  uint64_t* d_hreg = nullptr;   // [RENO_MAX_FRAMES + 1] hash region starts of a frame batch

  // model buffers (packed model rows: scale b at d_moff[b] ..)
  float* h_a = nullptr;         // [cap_rows][C]
  float* h_b = nullptr;
  float* h_c = nullptr;         // full predictor: X_A = Emb_O[O] of the parent scales (with a zero row)
  float* h_d = nullptr;         // full predictor: X_B of the target scales (with a zero row)
  int32_t* d_nbr = nullptr;     // [cap_rows][NBR_STRIDE]
  int32_t* d_perm = nullptr;    // [cap_rows] tile order of the conv layers after the first
  float* d_lse = nullptr;       // [cap_model] (two-stage head: stage 1)
  float* d_lse2 = nullptr;      // [cap_model] stage 2 of the two-stage head
  uint8_t* d_s1 = nullptr;      // [cap_model] S1 that stage 2 was evaluated with
  double* d_partial = nullptr;  // [NLEV][ceil(cap_pts / 64)] per-chunk bit sums
  double* d_total = nullptr;    // [NLEV]
  double* h_total = nullptr;    // pinned host mirror [NLEV]
  int32_t* h_count = nullptr;   // pinned host mirror [NLEV]
  uint32_t* h_err = nullptr;    // pinned host mirror [1]

  // packed weights (operand layouts of the conv/head kernels)
  float* w_conv[RENO_MAX_LAYERS] = {};
  float* w_bias[RENO_MAX_LAYERS] = {};
  float* w_head = nullptr;
  float* w_hbias = nullptr;
  float* w_head_plain = nullptr;  // [C][256] as given (two-stage: [C][H1 | H2]), for code lengths
  float* w_emb = nullptr;         // [16][C] Emb(S1) of the two-stage head
  float* w_head_t = nullptr;      // head transposed, one row per symbol: [256][C] (two-stage: [H1^T; H2^T])
  float* w_embo = nullptr;        // [256][C] Emb_O of the full predictor
  float* w_embd = nullptr;        // [8][C]   Emb_D of the full predictor
  bool have_weights = false;

  // frame state
  int B = 0;                    // bit depth of the current frame (0 = none)
  bool encoder = false;
  uint32_t have_level = 0;      // bit b: V_b built
  uint32_t have_codes = 0;      // bit b: O_b known
  uint32_t have_pred = 0;       // bit b: TOP evaluated on V_b (two-stage: stage 1)
  uint32_t have_pred2 = 0;      // bit b: stage 2 of the two-stage head evaluated
  int64_t npoints = 0;
  int frames = 1;               // frames batched in this frame's keys
  int fbits = 0;                // frame-id bits above the Morton bits (ceil(log2(frames)))
  // hash region table of the current frame batch, null for a single frame
  const uint64_t* hreg() const { return frames > 1 ? d_hreg : nullptr; }

  // kernel timing (reno_profile)
  uint32_t prof_mask = 0;
  std::vector<hipEvent_t> prof_pool;
  size_t prof_used = 0;
  std::vector<ProfRec> prof_recs;
  // events a timed conv launch binds to its dispatch (hipExtLaunchKernelGGL),
  // set by a dispatch-bound ProfScope and consumed by that launch
  hipEvent_t ext_start = nullptr, ext_stop = nullptr;

  // whole-frame coding staging, grown on demand (device: bitstream, stream
  // regions, stream bookkeeping, symbol tables, base voxels and codes;
  // pinned host: bitstream, base voxels)
  static constexpr int FC_DEV = 5, FC_HOST = 2;
  void* fc_dev[FC_DEV] = {};
  size_t fc_dev_bytes[FC_DEV] = {};
  void* fc_host[FC_HOST] = {};
  size_t fc_host_bytes[FC_HOST] = {};

  int64_t pyr_tiles = 0;    // max tiles of the pyramid pass
  int64_t exp_tiles = 0;    // max tiles of one expansion

  // look-back status layout: [sort passes][sort_tiles][RADIX] | [pyr_tiles][NLEV] | [NLEV][exp_tiles]
  uint32_t* st_sort(int pass) const { return d_status + (size_t)pass * sort_tiles * RADIX; }
  uint32_t* st_pyr() const { return d_status + (size_t)MAX_PASSES * sort_tiles * RADIX; }
  uint32_t* st_exp(int b) const {
    return st_pyr() + (size_t)pyr_tiles * NLEV + (size_t)b * exp_tiles;
  }

  int b0() const { return p.min_bit_depth; }
  int64_t lv(int b) const { return (int64_t)(b - p.min_bit_depth) * cap_pts; }
  bool top() const { return p.model_mode == RENO_MODEL_TOP; }
  // kernel size of the full predictor's convs (3 or 5) and its offsets
  int ks() const { return p.kernel_size == 5 ? 5 : 3; }
  int kvol() const { return ks() * ks() * ks(); }
  // neighbour-map row: 27 offsets + 5 padding, or 125 + 3
  int nbr_stride() const { return ks() == 5 ? 128 : NBR_STRIDE; }
  // the full predictor runs on streamed-weight kernels when its weights do
  // not fit the LDS-resident conv kernel (C above 32 or a 5x5x5 kernel)
  bool wide() const { return top() && (p.channels > 32 || ks() == 5); }
  // rows of the feature buffers: the model rows, the zero row cap_model and,
  // for the full predictor, the base scale
  int64_t cap_rows() const { return cap_model + 1 + (top() ? cap_pts : 0); }
  // buffer that holds the last conv layer's output (h_L), per the ping-pong
  float* hlast() const { return top() ? h_a : ((p.layers & 1) ? h_a : h_b); }
};

// Brackets the launches made during its lifetime with a pair of events when
// the kind is being profiled.
struct ProfScope {
  Ctx& c;
  int kind;
  bool bound;
  hipEvent_t start = nullptr, end = nullptr;
  // bound = the scope holds exactly one kernel launch, which takes the two
  // events as its dispatch start / end timestamps (hipExtLaunchKernelGGL):
  // the interval is then the kernel's execution, without the launch gap or
  // the inter-kernel barrier that events recorded between launches include
  ProfScope(Ctx& ctx, int k, bool bind = false) : c(ctx), kind(k), bound(bind) {
    if (!((c.prof_mask >> kind) & 1u) || c.prof_used + 2 > c.prof_pool.size()) return;
    start = c.prof_pool[c.prof_used++];
    end = c.prof_pool[c.prof_used++];
    if (bound) {
      c.ext_start = start;
      c.ext_stop = end;
    } else {
      (void)hipEventRecord(start, c.stream);
    }
    c.prof_recs.push_back(ProfRec{kind, start, end});
  }
  ~ProfScope() {
    if (!end) return;
    if (!bound) {
      (void)hipEventRecord(end, c.stream);
    } else if (c.ext_start == start) {  // no launch took the events: an empty interval
      (void)hipEventRecord(start, c.stream);
      (void)hipEventRecord(end, c.stream);
    }
    if (bound) c.ext_start = c.ext_stop = nullptr;
  }
};

// ---- kernel launchers (each enqueues on ctx.stream; return hipError_t) ----
hipError_t launch_zero(Ctx& c, void* const* ptrs, const size_t* bytes, int n);
hipError_t launch_quantize(Ctx& c, const float* pts, int64_t n, int B, int passes, const int64_t* frame_start,
                           int frames);
hipError_t launch_sort_pass(Ctx& c, const uint64_t* in, uint64_t* out, int64_t n, int pass);
hipError_t launch_pyramid(Ctx& c, const uint64_t* sorted, int64_t n, int B);
hipError_t launch_codes(Ctx& c, int B);
hipError_t launch_set_base(Ctx& c, const int32_t* xyz, const int32_t* frame_of, const uint8_t* codes, int64_t n,
                           int B);
// What a new frame clears, as (pointer, bytes) pairs: first the error word,
// the scale counts and the row offsets (CLEAR_SMALL entries, which the
// base-scale kernels write next), then histograms, tickets, look-back status
// and the hash.  Returns the number of entries (at most 8).
constexpr int CLEAR_SMALL = 3;
inline int frame_clear(const Ctx& c, void** ptr, size_t* bytes) {
  void* const p_[7] = {c.d_err, c.d_count, c.d_moff, c.d_hist, c.d_ticket, c.d_status, c.d_hash};
  const size_t n_[7] = {16,
                        sizeof(int32_t) * NLEV,
                        sizeof(int32_t) * (NLEV + 1),
                        sizeof(uint32_t) * MAX_PASSES * RADIX,
                        sizeof(uint32_t) * TICKETS,
                        sizeof(uint32_t) * (size_t)c.status_words,
                        sizeof(HashSlot) << c.hash_lg};
  for (int i = 0; i < 7; ++i) {
    ptr[i] = p_[i];
    bytes[i] = n_[i];
  }
  return 7;
}
// The frame's clear and the base scale in one launch, for a base scale of
// fewer than 256 voxels (clear_set_base_fits).
bool clear_set_base_fits(int64_t n);
hipError_t launch_clear_set_base(Ctx& c, const int32_t* xyz, const int32_t* frame_of, const uint8_t* codes,
                                 int64_t n);
hipError_t launch_expand(Ctx& c, int b, const uint8_t* codes, int B);
hipError_t launch_expand_noalloc(const uint64_t* keys, const uint8_t* codes, int64_t n,
                                 uint64_t* child_keys, int32_t* child_parent, int64_t cap_children,
                                 int32_t* first_child, int64_t* result, hipStream_t stream);
hipError_t launch_pack_weights(Ctx& c, const reno_weights& w);
hipError_t launch_model(Ctx& c, int b_lo, int b_hi, float* logits, bool second);
hipError_t launch_head2(Ctx& c, int b, const uint8_t* s1, float* logits2);
hipError_t launch_code_length(Ctx& c, int b_lo, int b_hi, float* bits);
hipError_t launch_symbol_freqs(Ctx& c, int b, uint16_t* freq);
hipError_t launch_symbol_freqs16(Ctx& c, int b, int stage, uint16_t* freq);
hipError_t launch_symbol_intervals(Ctx& c, int b_lo, int b_hi, uint16_t* iv);
hipError_t launch_symbol_cdf(Ctx& c, int b, int stage, uint16_t* start);
// the decoder's tables, entries start | f << 16 per symbol ([N][256] or
// [N][16]); scratch ([N][K] uint16) is used only by contexts whose head
// does not fit the register-resident table kernels
hipError_t launch_symbol_entries(Ctx& c, int b, int stage, uint32_t* entries, uint16_t* scratch);
hipError_t launch_coords(Ctx& c, int b, int32_t* xyz, uint64_t* keys);
hipError_t launch_copy_level_u8(Ctx& c, int b, uint8_t* out);
hipError_t launch_copy_level_i32(Ctx& c, int b, const int32_t* src, int32_t* out);
hipError_t launch_neighbor_map(Ctx& c, int b, int32_t* out);

// whole-frame entropy coder (k_code.hip)
int64_t rans_stream_bound(const Ctx& c, int sections, int L);
hipError_t launch_rans_encode(Ctx& c, const uint16_t* iv, int b_lo, int b_hi, int stages, int L, uint32_t* region,
                              uint32_t* lens, int64_t G);
hipError_t launch_rans_layout(Ctx& c, int b_lo, int b_hi, int stages, int L, int B, const uint32_t* lens,
                              int64_t G, int64_t* offs, uint32_t* out, int64_t cap_words, int64_t* total);
hipError_t launch_rans_pack(Ctx& c, const uint32_t* region, const uint32_t* lens, const int64_t* offs, int L,
                            int64_t G, const int64_t* total, const int32_t* xyz, uint32_t* out, int64_t cap_words);
hipError_t launch_rans_decode(Ctx& c, const uint32_t* words, int64_t nwords, int b, int L, int K,
                              const uint32_t* tab, const uint8_t* s1, uint8_t* out, uint64_t* fpos, int t,
                              int64_t p0, bool last);

// releases the whole-frame coding staging
void frame_free(Ctx& c);

}  // namespace reno

// the opaque handle of the C ABI
struct reno_ctx : reno::Ctx {};
