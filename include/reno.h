/*
 * reno.h - C ABI of the MI355X (gfx950) hot path of the RENO LiDAR geometry
 * codec (You et al., "RENO: Real-Time Neural Compression for 3D LiDAR Point
 * Clouds", CVPR 2025).
 *
 * The library turns one LiDAR frame into a multiscale sparse tensor
 * (Sec. 3, Eq. 1), derives the 8-bit occupancy code of every voxel (FOG,
 * Sec. 3.1), evaluates the target occupancy predictor on the occupied voxels
 * of each scale (TOP, Sec. 3.2, Eq. 5) to a 256-way distribution and an ideal
 * code length (Eq. 4), and on the decoder side expands codes into the next
 * scale (FCG, Sec. 3.1).  Arithmetic coding stays on the host; a host rANS
 * coder is exported for round-trip validation.
 *
 * Conventions (apply to every call unless stated otherwise):
 *  - Scales are bit depths.  A frame has scales b0 .. B (b0 = min_bit_depth,
 *    B = the frame's bit depth); scale b has N_b voxels V_b on a 2^b grid.
 *    Codes O_b exist for b0 <= b < B.  The model scales are b0 < b < B
 *    (Eq. 3 conditions O^d on scale d-1 for d = 1 .. D-1; the initial state
 *    (C^0, O^0) is coded raw).
 *  - Voxel order inside a scale is ascending Morton key
 *    key(x,y,z) = sum_i x_i 2^(3i) + y_i 2^(3i+1) + z_i 2^(3i+2), so that the
 *    children of v are 8*key(v) + delta with delta = dx + 2dy + 4dz (Eq. 8)
 *    and the sorted finer scale equals the FCG expansion order.
 *  - Array arguments are DEVICE pointers (hipMalloc or torch memory) unless
 *    the name ends in _host.  The caller owns them and keeps them alive until
 *    the context stream has passed the call.
 *  - Every call enqueues on the context's HIP stream and returns without
 *    waiting, except calls that write a _host value, which synchronise.
 *  - Sizes produced on the device (N_b) stay on the device; output buffers
 *    must hold the capacity stated for each call.
 *  - Errors are returned as reno_status, never thrown or aborted; the message
 *    is available from reno_last_error.  Data errors found by kernels
 *    (non-finite point, zero code, capacity overflow, ...) are latched on the
 *    device and reported by the next synchronising call (RENO_E_INPUT or
 *    RENO_E_CAPACITY); the frame's outputs are then undefined.
 *  - One context per stream; contexts are independent and may run
 *    concurrently on different streams.  A context is not thread-safe.
 */
#ifndef RENO_H
#define RENO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct reno_ctx reno_ctx;

typedef enum {
  RENO_OK = 0,
  RENO_E_INVALID = -1,  /* bad argument (null pointer, out-of-range scale or size) */
  RENO_E_STATE = -2,    /* call out of order (e.g. predict before the scale exists) */
  RENO_E_NOMEM = -3,    /* device allocation failed at create time */
  RENO_E_HIP = -4,      /* a HIP runtime call failed */
  RENO_E_CAPACITY = -5, /* a frame exceeded the capacities given at create time */
  RENO_E_INPUT = -6     /* bad data found on the device (non-finite point, zero
                           code, unsorted or duplicate base voxels) */
} reno_status;

#define RENO_MAX_LAYERS 8
#define RENO_SYMBOLS 256
#define RENO_KVOL 27
#define RENO_IN_FEATURES 11
#define RENO_MAX_BIT_DEPTH 21
#define RENO_ALL_SCALES (-1)
#define RENO_MAX_FRAMES 1024
#define RENO_HEAD_ONE_STAGE 0   /* one 256-way softmax over the code (Eq. 10) */
#define RENO_HEAD_TWO_STAGE 1   /* bitwise two-stage head (Eqs. 11-13) */
#define RENO_PREC_FP32 0        /* conv layers and heads on fp32 MFMA */
#define RENO_PREC_BF16X3 1      /* each fp32 operand split into bf16 hi + lo, products
                                   hi*hi + hi*lo + lo*hi on bf16 MFMA with fp32
                                   accumulation (~2^-16 relative per product) */
#define RENO_MODEL_PLAIN 0      /* 11 input bits [delta, parent code] (Eqs. 7-8), L sparse
                                   conv + ReLU layers (Eq. 9) */
#define RENO_MODEL_TOP 1        /* full target occupancy predictor (Sec. 3.2, Eqs. 6-9):
                                   Emb_O of the parent scale's codes and a residual block
                                   on the parent scale, replication + Emb_D of the octant
                                   and a residual block on the target scale; fp32 only */

/* Capacities and model shape, fixed for the life of a context. */
typedef struct {
  int64_t max_points;        /* raw points per frame; also the per-scale voxel capacity */
  int64_t max_model_voxels;  /* sum of N_b over the model scales; 0 selects
                                (max_bit_depth - min_bit_depth - 1) * max_points, which
                                always suffices; a tighter value saves memory and the
                                per-frame hash clear */
  int max_bit_depth;         /* largest B accepted, <= RENO_MAX_BIT_DEPTH (keys use 3B bits) */
  int min_bit_depth;         /* b0, the coarsest scale, 0 <= b0 < B */
  double range_m;            /* R: the grid covers [-R, R) on each axis */
  int in_features;           /* must be RENO_IN_FEATURES */
  int channels;              /* C: 16 or 32 */
  int layers;                /* L: 1 .. RENO_MAX_LAYERS sparse conv layers */
  int head_mode;             /* RENO_HEAD_ONE_STAGE (0) or RENO_HEAD_TWO_STAGE */
  int precision;             /* RENO_PREC_FP32 (0) or RENO_PREC_BF16X3 */
  int model_mode;            /* RENO_MODEL_PLAIN (0) or RENO_MODEL_TOP (layers is then
                                unused: the full predictor has its four convs) */
  int kernel_size;           /* full predictor: 3 (0 reads as 3) or 5; the plain model
                                uses 3.  Channels: 16 or 32 for the plain model; 16,
                                32, 64 or 128 for the full predictor (c128 with kernel
                                5 is the large variant) */
} reno_params;

/* Model weights (fp32, device memory, row-major).  Layout:
 *   conv_w[l]  [27][C_in][C]   C_in = 11 for l = 0, C otherwise;
 *              offset k = (dx+1) + 3(dy+1) + 9(dz+1)
 *   conv_b[l]  [C]
 *   head_w     [C][256]      one-stage head
 *   head_b     [256]
 * Two-stage head (Sec. 3.2, Eqs. 11-13; the code O splits into the first
 * sub-code S1 = O & 15, children delta 0..3, coded first, and S2 = O >> 4):
 *   head1_w    [C][16]   head1_b [16]   z1 = head1_w^T h + head1_b
 *   emb_s1     [16][C]                  Emb(S1), added to h before stage 2
 *   head2_w    [C][16]   head2_b [16]   z2 = head2_w^T (h + emb_s1[S1]) + head2_b
 * Full predictor (RENO_MODEL_TOP; conv_w / conv_b are then not read):
 *   emb_o      [256][C]  Emb_O, indexed by the code of a voxel of scale d-1
 *   emb_d      [8][C]    Emb_D, indexed by the octant delta of a voxel of scale d
 *   top_w[i]   [ks^3][C][C], top_b[i] [C]: convs A1, A2 (residual block on scale
 *              d-1) and B1, B2 (residual block on scale d); a block computes
 *              ReLU(x + conv2(ReLU(conv1(x)))) with biases inside both convs
 * Only the pointers of the context's model and head modes are read.        */
typedef struct {
  const float* conv_w[RENO_MAX_LAYERS];
  const float* conv_b[RENO_MAX_LAYERS];
  const float* head_w;
  const float* head_b;
  const float* head1_w;
  const float* head1_b;
  const float* emb_s1;
  const float* head2_w;
  const float* head2_b;
  const float* emb_o;
  const float* emb_d;
  const float* top_w[4];
  const float* top_b[4];
} reno_weights;

/* Creates a context on the current HIP device that enqueues on `hip_stream`
 * (a hipStream_t; NULL = the null stream).  Allocates every device buffer
 * the context needs for the given capacities; no later call allocates. */
reno_status reno_create(const reno_params* params, void* hip_stream, reno_ctx** out);
reno_status reno_destroy(reno_ctx* ctx);
/* Message of the last failed call on this context ("" if none).  With a NULL
 * context, the message of the last failed reno_create on this thread. */
const char* reno_last_error(const reno_ctx* ctx);
/* Waits for the context stream and reports latched device errors. */
reno_status reno_sync(reno_ctx* ctx);
/* Sizes fixed at create time, into info_host[4] (host memory): [0] coordinate
 * hash slots (16 bytes each), [1] look-back status words (4 bytes each), [2]
 * model-row capacity (max_model_voxels as resolved), [3] device bytes the
 * context allocated.  No device work. */
reno_status reno_memory_info(const reno_ctx* ctx, int64_t* info_host);

/* Copies the model weights into the context's operand layout (Sec. 3.2:
 * one parameter set shared by all scales).  Must precede predict_probs. */
reno_status reno_set_weights(reno_ctx* ctx, const reno_weights* w);

/* ENCODER (Sec. 3, Eq. 1; Sec. 3.1 FOG).  points: fp32 xyz [n][3].
 * Quantises each coordinate to the 2^bit_depth grid over [-R, R)
 * (u = ((p + R) * 2^B) / (2R) in fp64, floor, clamp to [0, 2^B - 1]),
 * removes duplicates, builds V_b for b = b0 .. B, the codes O_b for
 * b0 <= b < B (bit delta of O_b[v] set iff child 2v + delta is occupied) and
 * the parent links.  n may be 0.  Requires b0 < bit_depth <= max_bit_depth
 * and n <= max_points. */
reno_status reno_build_pyramid(reno_ctx* ctx, const float* points, int64_t n, int bit_depth);

/* DECODER start (Eq. 2: the initial state (C^0, O^0)).  Sets scale b0 of a
 * frame of bit depth `bit_depth` to the n voxels xyz int32 [n][3] (strictly
 * ascending Morton order, coordinates in [0, 2^b0)) with codes [n] (1..255). */
reno_status reno_set_base(reno_ctx* ctx, int bit_depth, const int32_t* xyz, const uint8_t* codes,
                          int64_t n);

/* FRAME BATCH (several independent frames coded as one, for throughput; each
 * frame is coded exactly as alone, Sec. 3 applied per frame).  The frames
 * share one key space: a scale-b voxel of frame f has the key
 * f << 3b | Morton(v), so frames never share a parent, a neighbour or a hash
 * slot, and every scale's launch covers all frames.  fb = ceil(log2(frames))
 * bits of frame id sit above the Morton bits; 3 * bit_depth + fb <= 63.
 *
 * Encoder: points of frame f are points[frame_start[f] .. frame_start[f+1])
 * (frame_start: device int64 [frames + 1], 0 = first <= ... <= last = n;
 * malformed ranges latch RENO_E_INPUT).  1 <= frames <= 1024.  Scale b then
 * holds every frame's voxels in (frame, Morton) order; coords return the
 * Morton part, the keys getter the full keys.  Code lengths add the raw
 * initial state of every frame (32 bits each for the counts).
 * Decoder: the base voxels carry their frame id (device int32 [n], in
 * (frame, Morton) strictly ascending order together with xyz; an id outside
 * [0, frames) latches RENO_E_INPUT); expand and predict then run on all
 * frames at once.  Device arrays are read on the context stream. */
reno_status reno_build_pyramid_frames(reno_ctx* ctx, const float* points, int64_t n,
                                      const int64_t* frame_start, int frames, int bit_depth);
reno_status reno_set_base_frames(reno_ctx* ctx, int bit_depth, const int32_t* xyz, const int32_t* frame_of,
                                 const uint8_t* codes, int64_t n, int frames);

/* DECODER step (Sec. 3.1 FCG).  Records O_scale := codes[N_scale] (codes may
 * be NULL when O_scale is already known, i.e. for the base scale after
 * set_base) and builds V_{scale+1} by keeping, for each voxel in order, the
 * children whose code bit is set, in ascending delta.  b0 <= scale < B;
 * V_scale must exist and V_{scale+1} must not (RENO_E_STATE otherwise; an
 * encoder context already holds every scale).  A zero code latches
 * RENO_E_INPUT. */
reno_status reno_expand(reno_ctx* ctx, int scale, const uint8_t* codes);

/* ALLOCATION-FREE FCG expansion, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  The decoder step of reno_expand (same kernel) on plain
 * arrays, without a context: each parent key in order emits 8*key + delta for
 * every set bit delta of its code, in ascending delta.  Allocates nothing:
 * its scratch (look-back status words, counters) is a static device array of
 * (64 + RENO_NOALLOC_MAX_PARENTS / 512) * 4 bytes (256 KiB) that each device
 * the library runs on holds until the process ends.
 *   keys          [n] parent keys (Morton keys, optionally with frame bits above
 *                 them), each below 2^61; their order is the output order
 *   codes         [n] occupancy codes, each in [1, 255]
 *   n             0 <= n <= RENO_NOALLOC_MAX_PARENTS
 *   child_keys    [cap_children] out: the children's keys
 *   child_parent  [cap_children] out: row of each child's parent in keys
 *   cap_children  capacity of both child arrays, 0 <= cap_children < 2^31
 *   first_child   [n] out, or NULL: row of each parent's first child
 *   result        [2] int64 out: [0] children written (the total, clamped to
 *                 cap_children), [1] RENO_OK, or RENO_E_CAPACITY when the
 *                 children exceed cap_children, or RENO_E_INPUT for a zero code
 *                 or a key of 2^61 or more (outputs then undefined)
 *   hip_stream    stream of the current device (NULL: the null stream); every
 *                 launch is enqueued there and the call returns without waiting
 * All arrays are device pointers on the current device.  Argument errors
 * return RENO_E_INVALID and launch errors RENO_E_HIP, with the message in
 * reno_last_error(NULL) of the calling thread.  Every call on a device shares
 * that device's scratch (cleared at the start of each call): calls that
 * overlap on one device, on different streams, race and must be ordered by
 * the caller. */
#define RENO_NOALLOC_MAX_PARENTS (1 << 25)
#define RENO_NOALLOC_MAX_DEVICES 64
reno_status reno_expand_noalloc(const uint64_t* keys, const uint8_t* codes, int64_t n,
                                uint64_t* child_keys, int32_t* child_parent, int64_t cap_children,
                                int32_t* first_child, int64_t* result, void* hip_stream);

/* Number of voxels of a scale (synchronises). */
reno_status reno_num_voxels(reno_ctx* ctx, int scale, int64_t* n_host);
/* N_b of every scale in one copy: counts_host[b] for b = 0 .. RENO_MAX_BIT_DEPTH
 * (0 for scales not built); synchronises. */
reno_status reno_scale_counts(reno_ctx* ctx, int64_t* counts_host);
/* Voxels of a scale: xyz int32 [N][3] and/or Morton keys uint64 [N] (either may be NULL). */
reno_status reno_coords(reno_ctx* ctx, int scale, int32_t* xyz, uint64_t* keys);
/* Occupancy codes O_scale uint8 [N_scale], b0 <= scale < B (Eq. 1). */
reno_status reno_occupancy_codes(reno_ctx* ctx, int scale, uint8_t* codes);
/* Row of each voxel's parent in scale-1, int32 [N_scale] (-1 at b0). */
reno_status reno_parent_rows(reno_ctx* ctx, int scale, int32_t* parent);

/* TOP (Sec. 3.2, Eq. 5, in the configured form): on the voxels of `scale`
 * (b0 < scale < B), input features [delta bits 0..2, bits 0..7 of the parent's
 * code] (target embedding, Eqs. 7-8), L submanifold 3x3x3 sparse conv + ReLU
 * layers on the target coordinates (Eq. 9), a linear head to 256 logits and
 * the softmax normaliser (Eq. 10; 256 classes indexed by code value).
 * Needs V_scale and O_{scale-1}; does NOT need O_scale, so a decoder calls it
 * before the codes of the scale are known.  RENO_ALL_SCALES runs every model
 * scale in one batch (all scales must exist).  logits: optional fp32
 * [N_scale][256] (for RENO_ALL_SCALES, the scales concatenated in increasing
 * order).  weights: NULL uses the weights of the last reno_set_weights;
 * otherwise they are set first.
 * Two-stage head: stage 1 (16 logits over S1) always; stage 2 as well when
 * O_scale is known (an encoder context), with S1 = O_scale & 15.  logits is
 * then [N_scale][32]: the 16 stage-1 logits, then the 16 stage-2 logits
 * (left untouched when stage 2 does not run). */
reno_status reno_predict_probs(reno_ctx* ctx, int scale, const reno_weights* weights, float* logits);

/* Stage 2 of the two-stage head (Eq. 13) for a decoder that has decoded S1:
 * s1 uint8 [N_scale] (values 0..15; device memory) or NULL to take
 * S1 = O_scale & 15 when O_scale is known.  Needs predict_probs of the scale
 * (it reuses the features of the last conv layer).  logits2: optional fp32
 * [N_scale][16].  Values of s1 above 15 latch RENO_E_INPUT.  RENO_E_STATE in
 * a one-stage context. */
reno_status reno_predict_second(reno_ctx* ctx, int scale, const uint8_t* s1, float* logits2);

/* Ideal code length (Eq. 4): for a model scale, bits_v = -log2 p(O_scale[v])
 * under the distribution of the last predict_probs of that scale (two-stage
 * head: -log2 P(S1) - log2 P(S2 | S1), which needs stage 2 of the scale); for
 * scale == b0 the raw cost of the initial state, 32 + N_b0 * (3*b0 + 8) bits.
 * bits_per_voxel: optional fp32 [N_scale] (NULL for b0).  total_host:
 * optional, synchronises; the sum in double.  RENO_ALL_SCALES: the whole
 * frame (base + every model scale); bits_per_voxel then holds the model
 * scales concatenated. */
reno_status reno_code_length(reno_ctx* ctx, int scale, float* bits_per_voxel, double* total_host);

/* Neighbour map of a model scale, int32 [N_scale][ks^3] (ks = 3, or the full
 * predictor's kernel size): entry k is the row in V_scale of v + (dx,dy,dz),
 * k = (dx+h) + ks(dy+h) + ks^2(dz+h) with h = ks/2 (for ks = 3: (dx+1) +
 * 3(dy+1) + 9(dz+1)), or -1 when absent or outside [0, 2^scale)^3.
 * Available after predict_probs of that scale. */
reno_status reno_neighbor_map(reno_ctx* ctx, int scale, int32_t* map);

/* Quantised distribution for the host coder, uint16 [N_scale][256]:
 * f_s = 1 + floor(p_s * 65024) with p_s = exp(z_s - lse) in fp32, and the
 * 65536 - sum leftover added to the lowest-index largest f_s (so sum f = 2^16).
 * Deterministic: an encoder and a decoder context that computed the same
 * distribution produce identical tables. */
reno_status reno_symbol_freqs(reno_ctx* ctx, int scale, uint16_t* freq);
/* Two-stage head: the same rule over 16 symbols, f_s = 1 + floor(p_s * 65504)
 * (2^16 - 2*16), uint16 [N_scale][16]; stage 1 after predict_probs, stage 2
 * (given the S1 of the last stage-2 evaluation) after predict_second.  In
 * general for K symbols: f_s = 1 + floor(p_s * (2^16 - 2K)). */
reno_status reno_symbol_freqs16(reno_ctx* ctx, int scale, int stage, uint16_t* freq);
/* Encoder side of the same tables without shipping them: for each voxel the
 * interval (start = sum of f below the symbol, f) of its code in its table,
 * uint16 [N][2] (one-stage) or [N][4] (two-stage: S1 in the stage-1 table,
 * then S2 in the stage-2 table).  Needs the codes and predict_probs (and
 * stage 2).  RENO_ALL_SCALES: every model scale, concatenated in order. */
reno_status reno_symbol_intervals(reno_ctx* ctx, int scale, uint16_t* iv);
/* Decoder side in cumulative form: for each voxel of the scale the start of
 * every symbol in its table (start_s = sum of f_t for t < s, so start_0 = 0 and
 * f_s = start_{s+1} - start_s with start_K = 2^16), uint16 [N_scale][256] for
 * the one-stage head (stage 0), [N_scale][16] for stage 1 or 2 of the
 * two-stage head; the same tables as reno_symbol_freqs(16), summed on the
 * device.  Preconditions as for those calls. */
reno_status reno_symbol_cdf(reno_ctx* ctx, int scale, int stage, uint16_t* start);

/* Host rANS coder (Duda, arXiv:1311.2540) for one scale's stream; HOST
 * pointers.  64-bit state in [2^31, 2^63), 32-bit renormalisation words.
 * encode: symbols sym[n], frequency tables freq [n][256] (sum 2^16); writes at
 * most cap words to out and their count to *nwords_host.  decode: the
 * inverse; fails with RENO_E_INPUT on a corrupt or truncated stream. */
reno_status reno_rans_encode(const uint8_t* sym, const uint16_t* freq, int64_t n, uint32_t* out,
                             int64_t cap, int64_t* nwords_host);
/* rANS encode from intervals (host memory): iv[i * stride] = start,
 * iv[i * stride + 1] = frequency of symbol i (start + f <= 2^16); same
 * stream format as reno_rans_encode. */
reno_status reno_rans_encode_intervals(const uint16_t* iv, int64_t n, int64_t stride, uint32_t* out,
                                       int64_t cap, int64_t* nwords_host);
/* Decoding with 16-symbol tables freq [n][16] (the two-stage head). */
reno_status reno_rans_decode16(const uint32_t* in, int64_t nwords, const uint16_t* freq, int64_t n,
                               uint8_t* sym);
reno_status reno_rans_decode(const uint32_t* in, int64_t nwords, const uint16_t* freq, int64_t n,
                             uint8_t* sym);

/* Interleaved multi-stream form of the same coder (host memory), for coding
 * one scale on several host threads: symbol i goes to stream i mod S (S =
 * nstreams, 1 .. RENO_RANS_MAX_STREAMS), and each stream is exactly the
 * single-stream coding of its symbols (the format of reno_rans_encode).
 * encode: intervals as reno_rans_encode_intervals; the S streams are written
 * back to back to out (at most cap words in all) and their word counts to
 * nwords_host [S].  decode: the S streams back to back in `in` with their
 * counts, and the cumulative tables start [n][k] (k = 256 or 16, from
 * reno_symbol_cdf) instead of frequencies, so that no table is summed on the
 * host; writes sym [n].  threads = host threads to use (0: up to 16 of the
 * available cores); the threads belong to a pool the library keeps for the
 * life of the process.  Errors as for the single-stream calls. */
#define RENO_RANS_MAX_STREAMS 256
reno_status reno_rans_encode_streams(const uint16_t* iv, int64_t n, int64_t stride, int nstreams, int threads,
                                     uint32_t* out, int64_t cap, int64_t* nwords_host);
reno_status reno_rans_decode_streams(const uint32_t* in, const int64_t* nwords_host, int nstreams, int threads,
                                     const uint16_t* start, int k, int64_t n, uint8_t* sym);

/* WHOLE-FRAME CODING: the codec of Sec. 3 with the arithmetic coder of
 * Sec. 4.2 realised as rANS (the stream format of reno_rans_encode), one
 * frame's points to a self-describing bitstream and back in one call each,
 * every step on the GPU.
 * encode: points device float [n][3] as for reno_build_pyramid; builds the
 * pyramid, evaluates the model on every model scale, takes the symbol
 * intervals and codes each model scale (and each stage of the two-stage
 * head) as S = ceil(N_b / stream_symbols) interleaved streams, one wavefront
 * per stream (1 <= stream_symbols <= 65533).  Copies the bitstream to the
 * HOST array out (at most cap_words words) and its length to *nwords_host
 * (also when it fails with RENO_E_CAPACITY because cap_words is too small).
 * The context then holds the frame as after build_pyramid + predict_probs.
 * decode: the bitstream in HOST memory; copies it to the device once and
 * rebuilds V_b0 .. V_B scale by scale (expand, predict, cumulative tables,
 * one wavefront per stream decoding the scale's codes) without waiting on the
 * host, so that reno_coords(ctx, B, ...) afterwards returns the decoded
 * voxels.  Fails with RENO_E_INPUT on a bitstream that is not well formed
 * (bad magic, sizes out of range, a stream that ends early or does not end
 * in the coder's initial state, words left over, a zero code), or that was
 * made with another min_bit_depth or head; RENO_E_CAPACITY when its frame
 * exceeds the context's capacities.
 * Both need min_bit_depth <= 8 and weights set, and synchronise the context
 * stream (also when they fail after enqueuing work); device and pinned host
 * staging is allocated by the first call that needs it (and grown by later
 * ones) and kept until reno_destroy.
 * Bitstream (uint32 words): 0x4F4E4552, B, b0, stages (1 or 2),
 * stream_symbols L, N_b0; the base voxels bit-packed from the lowest bit up
 * as fields x | y << b0 | z << 2 b0 | code << 3 b0 of 3 b0 + 8 bits, padded
 * to a word; then for each model scale b0 < b < B in order and each stage:
 * the S stream lengths in words as 16-bit fields (two per word, the even
 * stream in the low half), then the S streams, stream j coding the scale's
 * voxels j, j + S, ... (an empty scale has one stream of two words). */
reno_status reno_encode_frame(reno_ctx* ctx, const float* points, int64_t n, int bit_depth, int stream_symbols,
                              uint32_t* out, int64_t cap_words, int64_t* nwords_host);
reno_status reno_decode_frame(reno_ctx* ctx, const uint32_t* in, int64_t nwords);

/* Kernel timing for measurement.  While a kind's bit is set in `kind_mask`,
 * every launch of that kind is bracketed by two HIP events recorded on the
 * context stream (event pairs come from a pool created by this call; launches
 * beyond the pool are not timed); the plain model's conv launches take the
 * two events as their own dispatch start and end (hipExtLaunchKernelGGL), so
 * those intervals are kernel execution alone.  reno_profile resets the accumulators;
 * reno_profile_read synchronises and returns, per kind, the summed
 * event-to-event milliseconds and the number of timed launches (arrays of
 * RENO_K_COUNT).  Launches captured into a HIP graph are not timed. */
typedef enum {
  RENO_K_ZERO = 0,      /* per-frame clear of counters, look-back state and hash */
  RENO_K_QUANTIZE,      /* quantisation, Morton keys, digit histograms */
  RENO_K_SORT,          /* one radix-sort pass */
  RENO_K_PYRAMID,       /* all scales, parents, first children, hash inserts */
  RENO_K_CODES,         /* FOG codes and layer-1 input bits */
  RENO_K_SET_BASE,      /* decoder initial state */
  RENO_K_EXPAND,        /* FCG expansion of one scale */
  RENO_K_CONV_FIRST,    /* first conv layer with the hash probes */
  RENO_K_CONV_MID,      /* a middle conv layer */
  RENO_K_CONV_LAST,     /* last conv layer fused with the 256-way head and softmax normaliser */
  RENO_K_CODE_LENGTH,   /* ideal bits and per-scale sums */
  RENO_K_OTHER,         /* weight packing, getters, symbol tables */
  RENO_K_TOP_INPUT,     /* full predictor: neighbour maps and embedding inputs */
  RENO_K_ENTROPY,       /* whole-frame coding: rANS streams, their layout, base packing */
  RENO_K_COUNT
} reno_kernel;

reno_status reno_profile(reno_ctx* ctx, uint32_t kind_mask);
reno_status reno_profile_read(reno_ctx* ctx, double* ms_host, int64_t* launches_host);

#ifdef __cplusplus
}
#endif
#endif /* RENO_H */
