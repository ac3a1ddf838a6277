// Target occupancy predictor (Sec. 3.2, Eq. 5) on gfx950, in the configured
// form: per voxel of a scale, the 11 input bits [delta, parent code] (target
// embedding, Eqs. 7-8), L submanifold 3x3x3 sparse conv + ReLU layers on the
// target coordinates (Eq. 9) and a linear head to 256 logits with the softmax
// normaliser (Eq. 10).
//
// Work unit: a wavefront owns a tile of 16 consecutive voxels of one scale (in
// launches of at most 4 tiles per block, a quad of waves shares it).
// Each layer is computed transposed, out^T[c_out][16] = sum_k W_k^T in_k^T, on
// fp32 MFMA 16x16x4: the A operand is the offset's weights (staged once per
// block in LDS, pre-swizzled so each lane reads its operands with 128-bit
// loads), the B operand is the gathered neighbour rows (each lane loads a
// contiguous slice of one neighbour row).  Only offsets with at least one
// occupied neighbour in the tile are issued.  The accumulator layout of the
// last conv layer is exactly the B operand layout of the head, so the head
// (16 x 256 logits per tile) runs from registers, followed by a row max / sum
// of exp over the 64 logits a lane holds and the 4 lanes sharing a voxel.
// Output-stationary: no atomics, a fixed summation order per voxel (4 offset
// groups, each chained from zero and folded onto the bias in group order; the
// softmax normaliser merged per 64-symbol group in group order), so an encoder
// and a decoder evaluating the same scale get bit-identical results whether a
// tile is computed by one wave (large launches) or split over a quad of waves
// by offset group and symbol group (launches of at most 4 tiles per block).

#include <type_traits>

#include "ctx.h"

namespace reno {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf8 __attribute__((ext_vector_type(8)));

constexpr int CONV_THREADS = 1024;
constexpr int CONV_WAVES = CONV_THREADS / 64;

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---- split-bf16 arithmetic (precision RENO_PREC_BF16X3) ----
// An fp32 operand x is carried as hi = bf16(x) and lo = bf16(x - hi) (both
// round to nearest even), so x = hi + lo to about 2^-16 relative; a product
// is taken as hi*hi + hi*lo + lo*hi (the lo*lo term, ~2^-16 relative, is
// dropped) on v_mfma_f32_16x16x32_bf16 with fp32 accumulation.  Operands
// travel as 8 bf16 packed in a uint4 (lane l: row/column l % 16, K slots
// 8 (l / 16) .. 8 (l / 16) + 7).
__device__ __forceinline__ f4 mfma_bf(const uint4& a, const uint4& b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf8, a), __builtin_bit_cast(bf8, b),
                                                 c, 0, 0, 0);
}
__device__ __forceinline__ uint32_t bf_bits(__bf16 h) { return __builtin_bit_cast(uint16_t, h); }
// hi and lo words of two floats (x0 in the low half)
__device__ __forceinline__ void split2(float x0, float x1, uint32_t& hi, uint32_t& lo) {
  const __bf16 h0 = (__bf16)x0, h1 = (__bf16)x1;
  const __bf16 l0 = (__bf16)(x0 - (float)h0), l1 = (__bf16)(x1 - (float)h1);
  hi = bf_bits(h0) | (bf_bits(h1) << 16);
  lo = bf_bits(l0) | (bf_bits(l1) << 16);
}
// split of 8 floats into packed hi / lo operands
__device__ __forceinline__ void split8(const float (&x)[8], uint4& hi, uint4& lo) {
  split2(x[0], x[1], hi.x, lo.x);
  split2(x[2], x[3], hi.y, lo.y);
  split2(x[4], x[5], hi.z, lo.z);
  split2(x[6], x[7], hi.w, lo.w);
}
// hi*hi + hi*lo + lo*hi accumulated into c
__device__ __forceinline__ f4 mfma_bf3(const uint4& ah, const uint4& al, const uint4& bh, const uint4& bl, f4 c) {
  c = mfma_bf(ah, bh, c);
  c = mfma_bf(ah, bl, c);
  return mfma_bf(al, bh, c);
}

// ---------------------------------------------------------------------------
// Weight packing.  Conv layer (C_in -> C): KS = ceil(C_in/4) MFMA k-steps per
// offset; lane l (g = l/16) feeds input channel ci = g*KS + s at step s and
// output channel co = 16*cb + l%16.  Packed [27][C/16][64][KSP], KSP = KS
// rounded up to 4, zero padded (kv offsets: 27, or 125 for a 5x5x5 kernel).
__global__ void k_pack_conv(const float* __restrict__ W, int c_in, int C, int KS, int KSP, int kv,
                            float* __restrict__ out) {
  const int ncb = C / 16;
  const int total = kv * ncb * 64 * KSP;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int s = i % KSP;
    const int lane = (i / KSP) % 64;
    const int cb = (i / (KSP * 64)) % ncb;
    const int k = i / (KSP * 64 * ncb);
    const int ci = (lane >> 4) * KS + s;
    const int co = cb * 16 + (lane & 15);
    out[i] = (s < KS && ci < c_in) ? W[((size_t)k * c_in + ci) * C + co] : 0.0f;
  }
}

// Conv weights W [kv][C][C] for the streamed-weight kernel: the operands of
// k_pack_conv (lane (r, g), step s = 4q + e: W[ci = g*KS + s][co = 16cb + r],
// KS = C/4), stored lane-fastest as 16-byte words [kv][C/16][KS/4][64], so a
// wave's LDS reads of one (cb, q) are 64 consecutive words (no bank conflicts).
__global__ void k_pack_conv_wide(const float* __restrict__ W, int C, int kv, float* __restrict__ out) {
  const int ncb = C / 16, KS = C / 4, nq = KS / 4;
  const int total = kv * C * C;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int e = i % 4;
    const int lane = (i / 4) % 64;
    const int q = (i / 256) % nq;
    const int cb = (i / (256 * nq)) % ncb;
    const int k = i / (256 * nq * ncb);
    const int ci = (lane >> 4) * KS + 4 * q + e;
    const int co = cb * 16 + (lane & 15);
    out[i] = W[((size_t)k * C + ci) * C + co];
  }
}

// Head H [C][NS] (NS = 256, or 16 per stage of the two-stage head): step
// t = 4*cb + r carries channel c = 16*cb + 4*g + r (the conv accumulator
// register r of column block cb); lane l carries symbol 16*sb + l%16.
// Packed [NS/16][64][C/4].
__global__ void k_pack_head(const float* __restrict__ H, int C, int NS, float* __restrict__ out) {
  const int KT = C / 4;
  const int total = NS / 16 * 64 * KT;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int t = i % KT;
    const int lane = (i / KT) % 64;
    const int sb = i / (KT * 64);
    const int c = 16 * (t >> 2) + 4 * (lane >> 4) + (t & 3);
    out[i] = H[(size_t)c * NS + sb * 16 + (lane & 15)];
  }
}

// bf16x3 conv weights: per (offset k, column block cb, lane (r, g)) the A
// operand W^T[co = 16cb + r][ci = 8g + j], j = 0..7 (zero for ci >= c_in),
// as 4 words of hi then 4 words of lo.  Packed [27][C/16][64][8] uint32.
__global__ void k_pack_conv_bf(const float* __restrict__ W, int c_in, int C, uint32_t* __restrict__ out) {
  const int ncb = C / 16;
  const int total = 27 * ncb * 64 * 4;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int pr = i % 4;                 // pair of K slots
    const int lane = (i / 4) % 64;
    const int cb = (i / 256) % ncb;
    const int k = i / (256 * ncb);
    const int co = cb * 16 + (lane & 15);
    float x[2];
    for (int h = 0; h < 2; ++h) {
      const int ci = 8 * (lane >> 4) + 2 * pr + h;
      x[h] = ci < c_in ? W[((size_t)k * c_in + ci) * C + co] : 0.0f;
    }
    uint32_t hi, lo;
    split2(x[0], x[1], hi, lo);
    uint32_t* o = out + ((size_t)(k * ncb + cb) * 64 + lane) * 8;
    o[pr] = hi;
    o[4 + pr] = lo;
  }
}

// bf16x3 head H [C][NS]: per symbol block sb and lane (r, g) the A operand
// H[c(g, j)][16 sb + r] with the K slot -> channel map c(g, j) = 16 (j / 4) +
// 4g + (j % 4), which is the channel that register j % 4 of accumulator block
// j / 4 holds in lane (r, g) of the last conv layer (zero beyond C).  Packed
// [NS/16][64][8] uint32 (hi words, then lo words).
__global__ void k_pack_head_bf(const float* __restrict__ H, int C, int NS, uint32_t* __restrict__ out) {
  const int total = NS / 16 * 64 * 4;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int pr = i % 4;
    const int lane = (i / 4) % 64;
    const int sb = i / 256;
    const int sym = sb * 16 + (lane & 15);
    float x[2];
    for (int h = 0; h < 2; ++h) {
      const int j = 2 * pr + h;
      const int c = 16 * (j >> 2) + 4 * (lane >> 4) + (j & 3);
      x[h] = c < C ? H[(size_t)c * NS + sym] : 0.0f;
    }
    uint32_t hi, lo;
    split2(x[0], x[1], hi, lo);
    uint32_t* o = out + ((size_t)sb * 64 + lane) * 8;
    o[pr] = hi;
    o[4 + pr] = lo;
  }
}

// Transposes H [C][NS] into rows row0 .. row0+NS-1 of a [*][C] table.
__global__ void k_transpose_head(const float* __restrict__ H, int C, int NS, int row0, float* __restrict__ out) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < C * NS; i += gridDim.x * blockDim.x) {
    const int c = i / NS, s = i % NS;
    out[(size_t)(row0 + s) * C + c] = H[i];
  }
}

// Copies H [C][16] into columns col0 .. col0+15 of a [C][32] table.
__global__ void k_put_cols16(const float* __restrict__ H, int C, int col0, float* __restrict__ out) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < C * 16; i += gridDim.x * blockDim.x)
    out[(i / 16) * 32 + col0 + (i % 16)] = H[i];
}

// ---------------------------------------------------------------------------
// Two-stage head pieces, shared by the last conv layer (encoder: S1 known)
// and the decoder's stage-2 kernel, so both produce identical bits.
//
// 16 logits of one packed symbol block for a tile: lane (r, g) ends with the
// logits of symbols 4g .. 4g+3 of voxel r.  h is the tile's feature block in
// the accumulator layout (lane (r, g), register e of block q: channel
// 16q + 4g + e of voxel r).
template <int C>
__device__ __forceinline__ f4 head16(const f4* __restrict__ hp, const float* __restrict__ hb, const f4 (&h)[C / 16],
                                     int g) {
  f4 zz = *reinterpret_cast<const f4*>(hb + 4 * g);
#pragma unroll
  for (int q = 0; q < C / 16; ++q) {
    const f4 hv = hp[q];
#pragma unroll
    for (int e = 0; e < 4; ++e) zz = mfma4(hv[e], h[q][e], zz);
  }
  return zz;
}

// Natural-log normaliser of the 16 logits spread over lanes r, r+16, r+32, r+48.
__device__ __forceinline__ float lse16(const f4& z) {
  float m = fmaxf(fmaxf(z[0], z[1]), fmaxf(z[2], z[3]));
  m = fmaxf(m, __shfl_xor(m, 16));
  m = fmaxf(m, __shfl_xor(m, 32));
  float s = (__expf(z[0] - m) + __expf(z[1] - m)) + (__expf(z[2] - m) + __expf(z[3] - m));
  s += __shfl_xor(s, 16);
  s += __shfl_xor(s, 32);
  return m + __logf(s);
}

// B operand of the bf16x3 head from the accumulator layout (K slot j of lane
// (r, g) = register j % 4 of block j / 4; zero beyond C).
template <int C>
__device__ __forceinline__ void head_operand_bf(const f4 (&h)[C / 16], uint4& hi, uint4& lo) {
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (j / 4 < C / 16) ? h[j / 4 < C / 16 ? j / 4 : 0][j % 4] : 0.0f;
  split8(x, hi, lo);
}

// bf16x3 version of head16: hp points at this lane's packed words of the block.
template <int C>
__device__ __forceinline__ f4 head16_bf(const uint4* __restrict__ hp, const float* __restrict__ hb,
                                        const uint4& bh, const uint4& bl, int g) {
  f4 zz = *reinterpret_cast<const f4*>(hb + 4 * g);
  return mfma_bf3(hp[0], hp[1], bh, bl, zz);
}

// h + Emb(S1) in the accumulator layout (emb_row = emb_s1 + S1 * C).
template <int C>
__device__ __forceinline__ void add_emb(const f4 (&h)[C / 16], const float* __restrict__ emb_row, int g,
                                        f4 (&out)[C / 16]) {
#pragma unroll
  for (int q = 0; q < C / 16; ++q) {
    const f4 e = *reinterpret_cast<const f4*>(emb_row + 16 * q + 4 * g);
#pragma unroll
    for (int i = 0; i < 4; ++i) out[q][i] = h[q][i] + e[i];
  }
}

__global__ void k_copy_f32(const float* __restrict__ src, float* __restrict__ dst, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    dst[i] = src[i];
}

// ---------------------------------------------------------------------------
struct ConvArgs {
  int b_lo, b_hi, b0;
  const int32_t* count;
  const int32_t* moff;
  int64_t cap_pts, cap_model;
  const uint64_t* lv_key;
  const uint16_t* lv_feat;
  const HashSlot* hash;
  int hash_lg;
  const uint64_t* hreg;   // hash region starts of a frame batch (null: one frame)
  int32_t* nbr;           // [cap_model][NBR_STRIDE], entries 27.. are -1
  const float* h_in;      // [cap_model + 1][C_in], row cap_model all zero (unused by layer 1)
  int64_t zero_feat;      // index of a zero entry of lv_feat
  float* h_out;           // [cap_model][C]
  const float* w;         // packed conv weights
  const float* bias;      // [C]
  const float* hw;        // packed head weights (last layer)
  const float* hb;        // [256]
  float* lse;             // [cap_model]
  float* logits;          // optional [rows][256] (two-stage: [rows][32]), row = packed row - moff[b_lo]
  uint32_t* err;
  // two-stage head
  const float* emb;       // [16][C]
  const uint8_t* s1_code; // codes of the per-scale regions (S1 = O & 15), or NULL: stage 1 only
  float* lse2;            // [cap_model]
  uint8_t* s1_out;        // [cap_model] the S1 stage 2 used
  const int32_t* perm;    // optional tile order: tile slot -> packed row (layers after the first)
  // full predictor
  const float* res;       // residual input added before the ReLU (same rows as h_out), or NULL
  int b_ext;              // scale whose rows live past the zero row (the base scale), or -1
  int64_t ext_off;        // first packed row of that scale (cap_model + 1)
  int64_t cap_rows;       // rows of the feature buffers
  int fb;                 // frame-id bits above the Morton bits (frame batch), else 0
  // replication + octant embedding fused into the epilogue (Eqs. 7-8): each
  // voxel's result F, plus Emb_D[delta], goes to the rows of its children
  float* xb;              // child rows' input X_B (rows of scale b + 1), or NULL
  const float* emb_d;     // [8][C]
  const uint8_t* code;    // per-scale regions: O_b
  const int32_t* fc;      // per-scale regions: first child row in V_{b+1}
};

// Packed-row layout of the scales: scale b at moff[b] .. below the reserved
// zero row cap_model; the full predictor also models the base scale, whose
// rows sit past the zero row at ext_off.
struct RowMap {
  const int32_t* count;
  const int32_t* moff;
  int64_t cap_model;
  int b_ext;
  int64_t ext_off, cap_rows;
};

// First packed row and voxel count of scale b; a scale that would not fit
// reads as empty (the overflow was latched where its size was made).
__device__ __forceinline__ void scale_span(const RowMap& m, int b, int64_t& mo, int64_t& n) {
  n = m.count[b];
  if (b == m.b_ext) {
    mo = m.ext_off;
    if (mo + n > m.cap_rows) n = 0;
  } else {
    mo = m.moff[b];
    if (mo + n > m.cap_model) n = 0;
  }
}

// Entry j (wave-uniform) of the 8 neighbour rows a lane holds in two int4,
// as a branch-free select tree.
__device__ __forceinline__ int32_t pick8(const int4& lo, const int4& hi, int j) {
  const bool b0 = j & 1, b1 = j & 2, b2 = j & 4;
  const int32_t l01 = b0 ? lo.y : lo.x, l23 = b0 ? lo.w : lo.z;
  const int32_t h01 = b0 ? hi.y : hi.x, h23 = b0 ? hi.w : hi.z;
  const int32_t l = b1 ? l23 : l01, h = b1 ? h23 : h01;
  return b2 ? h : l;
}

// Copies n16 16-byte words from global memory to LDS, all loads of a thread
// issued before its stores.
template <int N16, int THREADS>
__device__ __forceinline__ void stage_lds(const f4* __restrict__ src, f4* dst, int tid) {
  constexpr int PER = (N16 + THREADS - 1) / THREADS;
  constexpr int BATCH = PER < 12 ? PER : 12;
#pragma unroll
  for (int b0 = 0; b0 < PER; b0 += BATCH) {
    f4 v[BATCH];
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int idx = (b0 + i) * THREADS + tid;
      if (b0 + i < PER && idx < N16) v[i] = src[idx];
    }
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int idx = (b0 + i) * THREADS + tid;
      if (b0 + i < PER && idx < N16) dst[idx] = v[i];
    }
  }
}

// Register-staged copy of N16 16-byte words into LDS, in two halves: the
// loads (issued early, so that their latency overlaps other work) and the
// stores.
template <int N16, int THREADS>
struct Staged {
  static constexpr int PER = (N16 + THREADS - 1) / THREADS;
  f4 v[PER];
  __device__ __forceinline__ void load(const f4* __restrict__ src, int tid) {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = i * THREADS + tid;
      if (idx < N16) v[i] = src[idx];
    }
  }
  __device__ __forceinline__ void store(f4* dst, int tid) const {
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int idx = i * THREADS + tid;
      if (idx < N16) dst[idx] = v[i];
    }
  }
};

// Neighbour rows of a voxel from the parent scale.  The 27 cells around v lie
// in at most 8 cells of the parent scale: the parent p and, per axis, the
// neighbour of p on v's side.  Lane (r, g) probes cells e = 2g and 2g+1
// (e = ex + 2ey + 4ez) of its voxel r; each hit gives the cell's code and
// first-child row, from which every neighbour row follows by the FCG order.
// par is the 8-entry LDS slot of voxel r (shared by the 4 lanes of r); the
// lane ends with the rows of offsets 8g .. 8g+7 (-1: absent or off-grid).
//
// The cells are stepped to directly on the Morton key (dilated-integer
// increments and decrements of one axis's bits), so no coordinate is ever
// unpacked; a step off the grid leaves the probe empty, and every neighbour
// in such a cell reads as absent, so the offsets need no bounds of their own.

// Per entry slot j of the 8 a lane holds, the four lane groups' offsets
// k = 8g + j packed one byte each: bit 6 the offset exists (k < 27), bits 3..5
// the axes it moves up, bits 0..2 the axes it moves at all (k = dx+1 +
// 3 (dy+1) + 9 (dz+1)).
__host__ __device__ constexpr uint32_t offset_moves(int j) {
  uint32_t v = 0;
  for (int g = 0; g < 4; ++g) {
    const int k = 8 * g + j;
    if (k < 27) {
      const int dx = k % 3 - 1, dy = (k / 3) % 3 - 1, dz = k / 9 - 1;
      const uint32_t nz = (dx != 0 ? 1u : 0u) | (dy != 0 ? 2u : 0u) | (dz != 0 ? 4u : 0u);
      const uint32_t up = (dx == 1 ? 1u : 0u) | (dy == 1 ? 2u : 0u) | (dz == 1 ? 4u : 0u);
      v |= (64u | (up << 3) | nz) << (8 * g);
    }
  }
  return v;
}

// One step of the cell with Morton key k (axis bits m) towards +1 (up) or -1
// along that axis; `off` is set when the step leaves the grid.
__device__ __forceinline__ uint64_t morton_step(uint64_t k, uint64_t m, bool up, bool& off) {
  const uint64_t a = k & m, rest = k & ~m;
  off = up ? a == m : a == 0ull;
  const uint64_t na = up ? ((a | ~m) + 1ull) & m : (a - 1ull) & m;
  return na | rest;
}

__device__ __forceinline__ void parent_cell_rows(uint64_t kf, int b, int g, const HashSlot* __restrict__ hash,
                                                 int hash_lg, const uint64_t* __restrict__ hreg, int fb,
                                                 volatile uint64_t* par, int32_t (&nb)[8]) {
  const uint64_t key = morton_part(kf, b), fr = frame_part(kf, b) << (3 * (b - 1));
  const uint32_t oct = (uint32_t)key & 7u;  // v's octant in its parent: the side of each neighbour cell
  const uint64_t pk = key >> 3;
  const uint64_t all = (1ull << (3 * (b - 1))) - 1ull;
  const uint64_t mx = 0x1249249249249249ull & all, my = (mx << 1) & all, mz = (mx << 2) & all;
  // lane group g probes cells 2g and 2g + 1: the y and z steps of g, then x
  bool off_y = false, off_z = false, off_x = false;
  uint64_t c0 = pk;
  if (g & 1) c0 = morton_step(c0, my, (oct & 2u) != 0u, off_y);
  if (g & 2) c0 = morton_step(c0, mz, (oct & 4u) != 0u, off_z);
  const uint64_t c1 = morton_step(c0, mx, (oct & 1u) != 0u, off_x);
  const bool ok0 = !(off_y || off_z), ok1 = ok0 && !off_x;
  uint64_t tk[2];
  tk[0] = ok0 ? tag_key(fr | c0, b - 1, fb) : 0ull;
  tk[1] = ok1 ? tag_key(fr | c1, b - 1, fb) : 0ull;
  uint2 hit[2];
  hash_find_n<2>(hash, hash_lg, hash_region(hreg, hash_lg, frame_part(kf, b)), tk, hit);
  // cross-lane exchange through LDS (volatile: every read goes to LDS)
  par[2 * g] = ((uint64_t)hit[0].y << 32) | hit[0].x;
  par[2 * g + 1] = ((uint64_t)hit[1].y << 32) | hit[1].x;
  __builtin_amdgcn_wave_barrier();
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t c = (offset_moves(j) >> (8 * g)) & 0xFFu;
    const uint32_t nz = c & 7u, up = (c >> 3) & 7u;
    // the parent-scale cell of the neighbour: a moved axis leaves v's parent
    // when the move points to v's side; its octant flips every moved axis
    const uint32_t e = nz & ~(oct ^ up), d = oct ^ nz;
    const uint64_t pc = par[e];
    const uint32_t first = (uint32_t)pc, code = (uint32_t)(pc >> 32);
    nb[j] = ((c & 64u) && ((code >> d) & 1u)) ? (int32_t)(first + __popc(code & ((1u << d) - 1u))) : -1;
  }
}

constexpr float LOG2E_F = 1.4426950408889634f;

// One group of 64 symbols of the 256-way head (symbol blocks 4 grp .. 4 grp
// + 3, 16 symbols each): logits z = H^T h + b on MFMA from the accumulator
// layout of h, stored when requested, and the group's normaliser terms per
// lane: gm = the max of the lane's 16 logits, part = the sum of exp(z - gm).
template <int C, bool BF>
__device__ __forceinline__ void head_group(const ConvArgs& a, const f4 (&acc)[C / 16], const float* s_h,
                                           const float* hb, int lane, int g, bool valid, int64_t prow,
                                           int64_t mo_first, int grp, float& gm, float& part) {
  constexpr int KT = C / 4;
  float* lo = (a.logits && valid) ? a.logits + (prow - mo_first) * 256 + 4 * g : nullptr;
  uint4 bh = make_uint4(0, 0, 0, 0), bl = bh;
  if constexpr (BF) head_operand_bf<C>(acc, bh, bl);
  f4 zz[4];
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4) {
    const int sb = grp * 4 + q4;
    if constexpr (BF) {
      zz[q4] = head16_bf<C>(reinterpret_cast<const uint4*>(s_h) + (sb * 64 + lane) * 2, hb + 16 * sb, bh, bl, g);
    } else {
      zz[q4] = *reinterpret_cast<const f4*>(hb + 16 * sb + 4 * g);
      const f4* hp = reinterpret_cast<const f4*>(s_h + (sb * 64 + lane) * KT);
#pragma unroll
      for (int q = 0; q < KT / 4; ++q) {
        const f4 hv = hp[q];
#pragma unroll
        for (int e = 0; e < 4; ++e) zz[q4] = mfma4(hv[e], acc[q][e], zz[q4]);
      }
    }
  }
  gm = zz[0][0];
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
    for (int e = 0; e < 4; ++e) gm = fmaxf(gm, zz[q4][e]);
  // exp(z - gm) as 2^(z log2(e) - gm log2(e)): one fused multiply-add per term
  const float gml = gm * LOG2E_F;
  part = __builtin_amdgcn_exp2f(fmaf(zz[0][0], LOG2E_F, -gml));
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4)
#pragma unroll
    for (int e = 0; e < 4; ++e)
      if (q4 || e) part += __builtin_amdgcn_exp2f(fmaf(zz[q4][e], LOG2E_F, -gml));
  if (lo) {
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) *reinterpret_cast<f4*>(lo + 16 * (grp * 4 + q4)) = zz[q4];
  }
}

// Running normaliser (m, s) of the logits seen so far, extended by a group
// with terms (gm, part); starts from (-inf, 0).
__device__ __forceinline__ void lse_merge(float& m, float& s, float gm, float part) {
  const float mn = fmaxf(m, gm);
  s = s * __expf(m - mn) + part * __expf(gm - mn);
  m = mn;
}

// The 4 lanes r, r+16, r+32, r+48 hold the 4 quarters of voxel r's symbols:
// merged by lane exchange, then lse = m + log(s) stored at row prow.
__device__ __forceinline__ void lse_finish(const ConvArgs& a, float m, float ssum, int g, bool valid, int64_t prow) {
#pragma unroll
  for (int o = 16; o <= 32; o <<= 1) {
    const float om = __shfl_xor(m, o), os = __shfl_xor(ssum, o);
    const float mn = fmaxf(m, om);
    ssum = ssum * __expf(m - mn) + os * __expf(om - mn);
    m = mn;
  }
  if (valid && g == 0) a.lse[prow] = m + __logf(ssum);
}

// Head of the last conv layer's features h (the conv accumulators of a tile:
// lane (r, g) holds channels 16 cb + 4 g .. + 3 of voxel r) in registers:
// the one-stage 256-way head with its softmax normaliser (Eq. 10), or the
// two-stage head (Eqs. 11-13).  Writes lse (lse2, S1) at row prow and, when
// requested, the logits at row prow - mo_first.
template <int C, bool TWO, bool BF>
__device__ __forceinline__ void head_epilogue(const ConvArgs& a, const f4 (&acc)[C / 16], const float* s_h, int lane,
                                              int g, bool valid, int64_t prow, int64_t mo, int64_t lvb,
                                              int64_t mo_first) {
  constexpr int KT = C / 4;
  constexpr int NCB = C / 16;
  if constexpr (TWO) {
    // ---- two-stage head (Eqs. 11-13): stage 1 over S1; stage 2 over S2
    // with h + Emb(S1) when the codes of the scale are known
    const f4* hp = reinterpret_cast<const f4*>(s_h) + lane * (KT / 4);
    const uint4* hpb = reinterpret_cast<const uint4*>(s_h) + lane * 2;
    f4 z1;
    if constexpr (BF) {
      uint4 bh, bl;
      head_operand_bf<C>(acc, bh, bl);
      z1 = head16_bf<C>(hpb, a.hb, bh, bl, g);
    } else {
      z1 = head16<C>(hp, a.hb, acc, g);
    }
    const float l1 = lse16(z1);
    if (valid && g == 0) a.lse[prow] = l1;
    float* lo = (a.logits && valid) ? a.logits + (prow - mo_first) * 32 + 4 * g : nullptr;
    if (lo) *reinterpret_cast<f4*>(lo) = z1;
    if (a.s1_code) {
      const int s1 = a.s1_code[lvb + (prow - mo)] & 15;
      f4 h2[NCB];
      add_emb<C>(acc, a.emb + s1 * C, g, h2);
      f4 z2;
      if constexpr (BF) {
        uint4 bh, bl;
        head_operand_bf<C>(h2, bh, bl);
        z2 = head16_bf<C>(hpb + 64 * 2, a.hb + 16, bh, bl, g);
      } else {
        z2 = head16<C>(hp + 64 * (KT / 4), a.hb + 16, h2, g);
      }
      const float l2 = lse16(z2);
      if (valid && g == 0) {
        a.lse2[prow] = l2;
        a.s1_out[prow] = (uint8_t)s1;
      }
      if (lo) *reinterpret_cast<f4*>(lo + 16) = z2;
    }
  }
  if constexpr (!TWO) {
    // ---- head: z^T[256][16] = H^T h^T with the conv accumulators as the B
    // operand, 64 symbols (4 blocks of 16) per group; the normaliser is
    // combined group by group in a fixed order (head_group / lse_merge), the
    // same order a tile split over several waves uses
    float m = -INFINITY, ssum = 0.0f;
#pragma unroll 1
    for (int grp = 0; grp < 4; ++grp) {
      float gm, part;
      head_group<C, BF>(a, acc, s_h, a.hb, lane, g, valid, prow, mo_first, grp, gm, part);
      lse_merge(m, ssum, gm, part);
    }
    lse_finish(a, m, ssum, g, valid, prow);
  }
}

// Tile of a block's slot, XCD-aware: workgroups are dealt round-robin to the
// 8 XCDs (block b runs on XCD b % 8), so chunks of tch consecutive tiles are
// dealt to the XCDs in turn and the blocks of one XCD sweep that XCD's chunks
// together: tiles that gather the same neighbour rows run on one L2 at about
// the same time.  Increasing in the slot for a fixed block.
__device__ __forceinline__ int64_t conv_tile(int64_t slot, int64_t tch) {
  const int64_t xcd = blockIdx.x & 7, j = blockIdx.x >> 3, nb = gridDim.x >> 3;
  const int64_t k = j + nb * slot;  // the XCD's k-th tile
  return ((k / tch) * 8 + xcd) * tch + k % tch;
}

// Offsets of group i of the conv's fixed summation order: k in [7i, 7i + 7),
// the last group [21, 27).
__device__ __forceinline__ uint32_t group_offsets(int i) {
  const int lo = 7 * i, hi = i < 3 ? 7 * i + 7 : 27;
  return ((1u << hi) - 1u) & ~((1u << lo) - 1u);
}

template <int C, bool FIRST, bool LAST, bool TWO, bool BF>
__global__ void __launch_bounds__(CONV_THREADS) k_conv(ConvArgs a) {
  constexpr int NCB = C / 16;
  constexpr int KS = FIRST ? 3 : C / 4;
  constexpr int KSP = (KS + 3) & ~3;
  constexpr int KT = C / 4;
  // packed weights per (offset, column block, lane): fp32 KSP floats, bf16x3 8 words
  constexpr int WSZ = 27 * NCB * 64 * (BF ? 8 : KSP);
  constexpr int HSZ = LAST ? (TWO ? 2 : 16) * 64 * (BF ? 8 : KT) : 4;
  // offsets per pipeline stage: the first layer's gathers are 2-byte words behind a
  // few MFMAs each, and a shallow pipeline measured fastest there
  constexpr int PCH = FIRST ? 2 : 3;
  struct Gath {                        // one gathered neighbour slice
    uint32_t word;                     // first layer: 11 input bits
    f4 v[FIRST ? 1 : KSP / 4];         // later layers, fp32: KS channels
  };
  struct GathB {                       // later layers, bf16x3: channels 8g .. 8g+7
    uint32_t word;
    uint4 hi, lo;
  };
  using G = typename std::conditional<BF, GathB, Gath>::type;
  __shared__ __attribute__((aligned(16))) float s_w[WSZ];
  __shared__ __attribute__((aligned(16))) float s_h[HSZ];
  // per wave: parent cells (code<<32|first), rows padded to 9 so that the 16 voxels' cells lie in
  // different banks
  __shared__ uint64_t s_par[FIRST ? CONV_WAVES : 1][16][9];
  // per wave: the tile's neighbour rows, voxel by voxel (32 entries, the last 5 are -1), so that
  // a lane reads the row of any offset directly (the last layer has no room for them); rows
  // padded to 36 words, so that the 16 voxels' entries of one offset lie in 16 different banks
  constexpr bool ROWS = FIRST && !LAST && !BF;
  constexpr int RW = 36;
  __shared__ int32_t s_rows[ROWS ? CONV_WAVES : 1][16][RW];
  __shared__ int64_t s_tpre[NLEV + 1];
  __shared__ int64_t s_nv[NLEV];   // N_b of the launch's scales
  __shared__ int64_t s_mo[NLEV];   // first packed row of each scale
  __shared__ int s_next;           // next dynamically handed-out tile slot of this block

  // the wave index through a lane read: the compiler then keeps the tile loop,
  // the offset sets and the group folds in scalar registers and branches
  const int tid = threadIdx.x, w = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int r = lane & 15, g = lane >> 4;
  const int nsc = a.b_hi - a.b_lo + 1;

  const RowMap rm{a.count, a.moff, a.cap_model, a.b_ext, a.ext_off, a.cap_rows};
  // Sizes of the launch's scales.  One scale: scalar loads.  Several (the
  // encoder's batched launch): all loaded at once, lane i of every wave
  // reading scale b_lo + i, and the tile prefix over the scales is a scan
  // across the lanes.  Lane i ends with scale i's rows (nb_l, mo_l), tiles
  // tl and inclusive tile prefix incl (0 and the total beyond the last scale).
  static_assert(NLEV < 32, "the scale scan covers 32 lanes");
  int64_t nb_l = 0, mo_l = 0, total_tiles;
  int tl = 0, incl;  // tiles of a scale and of a launch fit in 31 bits
  if (nsc == 1) {
    int64_t mo, nb;
    scale_span(rm, a.b_lo, mo, nb);
    total_tiles = (nb + 15) / 16;
    if (lane == 0) {
      nb_l = nb;
      mo_l = mo;
      tl = (int)total_tiles;
    }
    incl = (int)total_tiles;
  } else {
    if (lane < nsc) scale_span(rm, a.b_lo + lane, mo_l, nb_l);
    tl = (int)((nb_l + 15) / 16);
    incl = tl;
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    total_tiles = __builtin_amdgcn_readlane(incl, 31);  // uniform (scalar register)
  }
  // chunk size: 256 chunks per launch (32 per XCD) between 16 and 256 tiles
  const int64_t tch = total_tiles / 256 < 16 ? 16 : (total_tiles / 256 > 256 ? 256 : total_tiles / 256);
  // small launches: a quad of waves per tile (at most CONV_WAVES / 4 tiles per block)
  const bool quads = total_tiles <= (int64_t)gridDim.x * (CONV_WAVES / 4);  // uniform
  static_assert((16 * NCB * 64 * 16 + 16 * 64 * 8) <= WSZ * 4, "quad exchange area exceeds the weight area");
  if (quads ? (int64_t)blockIdx.x >= total_tiles : conv_tile(0, tch) >= total_tiles)
    return;  // whole block idle: no weight staging
  // weight and head loads of the whole block in one round trip
  Staged<WSZ / 4, CONV_THREADS> stw;
  Staged<LAST ? HSZ / 4 : 1, CONV_THREADS> sth;
  stw.load(reinterpret_cast<const f4*>(a.w), tid);
  if (LAST) sth.load(reinterpret_cast<const f4*>(a.hw), tid);
  if (w == 0 && lane <= NLEV) {
    if (lane == 0) s_next = 0;
    s_tpre[lane] = lane < nsc ? incl - tl : total_tiles;  // padding: never below a valid tile
    if (lane < NLEV) {
      s_nv[lane] = nb_l;
      s_mo[lane] = mo_l;
    }
  }
  stw.store(reinterpret_cast<f4*>(s_w), tid);
  if (LAST) sth.store(reinterpret_cast<f4*>(s_h), tid);
  __syncthreads();

  // A tile as the epilogue and the head need it.
  struct TileRef {
    int b;
    int64_t mo, prow, lvb;
    bool valid;
  };
  // Opens tile `tile` (scale, rows, neighbour rows) and accumulates it: grp < 0
  // gives the bias plus all 4 offset-group sums, folded in group order; grp in
  // 0 .. 3 gives that group's sum alone (a wave of a quad sharing the tile).
  auto conv_sum = [&](int64_t tile, int grp, TileRef& tr, f4 (&out)[NCB]) {
    int si = 0;  // scale of the tile: all prefix loads issued together
#pragma unroll
    for (int i = 1; i < NLEV; ++i) si += (s_tpre[i] <= tile) ? 1 : 0;
    const int b = a.b_lo + si;
    const int64_t nvox = s_nv[si];
    const int64_t mo = s_mo[si];
    const int64_t row = (tile - s_tpre[si]) * 16 + r;
    const bool valid = row < nvox;
    // idle lanes read a real row; with a tile order, slot -> row
    const int64_t pos = mo + (valid ? row : nvox - 1);
    const int64_t prow = (!FIRST && a.perm) ? (int64_t)a.perm[pos] : pos;
    const int64_t lvb = (int64_t)(b - a.b0) * a.cap_pts;

    // ---- neighbour rows: lane (r, g) holds offsets k = 8g .. 8g+7 of voxel r
    int4 nlo, nhi;
    if (FIRST) {
      int32_t nb[8];
      parent_cell_rows(a.lv_key[lvb + (prow - mo)], b, g, a.hash, a.hash_lg, a.hreg, a.fb, s_par[w][r], nb);
      nlo = make_int4(nb[0], nb[1], nb[2], nb[3]);
      nhi = make_int4(nb[4], nb[5], nb[6], nb[7]);
      if (valid && grp <= 0) {  // one wave of a quad stores the map rows
        int4* dst = reinterpret_cast<int4*>(a.nbr + prow * NBR_STRIDE + 8 * g);
        dst[0] = nlo;
        dst[1] = nhi;
      }
    } else {
      const int4* src = reinterpret_cast<const int4*>(a.nbr + prow * NBR_STRIDE + 8 * g);
      nlo = src[0];
      nhi = src[1];
    }
    if constexpr (ROWS) {
      int4* rr = reinterpret_cast<int4*>(&s_rows[w][r][8 * g]);
      rr[0] = nlo;
      rr[1] = nhi;
      __builtin_amdgcn_wave_barrier();
    }
    // occupied offsets of the tile: one ballot per entry slot j, lanes of
    // group g covering offsets 8g + j (the 5 padding entries are -1)
    uint32_t offs = 0;
    {
      const int32_t e8[8] = {nlo.x, nlo.y, nlo.z, nlo.w, nhi.x, nhi.y, nhi.z, nhi.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint64_t bal = __ballot(valid && e8[j] >= 0);
#pragma unroll
        for (int gg = 0; gg < 4; ++gg)
          offs |= ((bal >> (16 * gg)) & 0xFFFFull) ? (1u << (8 * gg + j)) : 0u;
      }
      offs &= 0x7FFFFFFu;
    }
    if (grp >= 0) offs &= group_offsets(grp);

    // ---- accumulate over the occupied offsets, software-pipelined: the
    // gathers of the next PCH offsets are issued before the MFMAs of the
    // current ones (double buffer; loads are never skipped, an unused slot
    // reads the zero row, so the wait counts stay exact).
    // Summation order per output: the offsets fall into 4 fixed groups
    // (k < 7, < 14, < 21, < 27); each group's products are chained on MFMA
    // from zero, in ascending offset order, and the 4 group sums are added to
    // the bias in group order: ((((bias + S0) + S1) + S2) + S3).
    f4 acc[NCB], tsum[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      tsum[cb] = *reinterpret_cast<const f4*>(a.bias + 16 * cb + 4 * g);
      acc[cb] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    int gcur = grp >= 0 ? grp : 0;  // group whose sum acc holds
    auto fold = [&]() {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        tsum[cb] += acc[cb];
        acc[cb] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      }
      ++gcur;
    };
    auto enter = [&](int k) {  // k: the next offset, wave-uniform
      while (k >= (gcur < 3 ? 7 * (gcur + 1) : 27)) fold();
    };
    auto take = [&](int (&ks)[PCH]) {
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        ks[c] = offs ? __builtin_ctz(offs) : -1;
        offs &= offs ? offs - 1u : 0u;
      }
    };
    auto gather = [&](const int (&ks)[PCH], G (&gb)[PCH]) {
      int32_t nn[PCH];
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        if constexpr (ROWS) nn[c] = s_rows[w][r][ks[c] & 31];
        else nn[c] = __shfl(pick8(nlo, nhi, ks[c] & 7), r + 16 * ((ks[c] & 31) >> 3));
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the exchanges back to back (one wait for all)
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        const int32_t n = (valid && ks[c] >= 0) ? nn[c] : -1;
        if constexpr (FIRST) {
          // absent neighbours read the reserved zero entry: no select on loaded data
          gb[c].word = n >= 0 ? a.lv_feat[lvb + n] : a.lv_feat[a.zero_feat];
        } else if constexpr (BF) {
          // rows hold [hi plane: C bf16][lo plane: C bf16]; lanes beyond C/8 feed zeros
          const int64_t srow = n >= 0 ? mo + n : a.cap_model;
          const uint4* src = reinterpret_cast<const uint4*>(a.h_in + srow * C);
          const int gq = g < C / 8 ? g : 0;
          gb[c].hi = src[gq];
          gb[c].lo = src[C / 8 + gq];
          if (g >= C / 8) gb[c].hi = gb[c].lo = make_uint4(0, 0, 0, 0);
        } else {
          // absent neighbours read the reserved all-zero row cap_model
          const int64_t srow = n >= 0 ? mo + n : a.cap_model;
          const f4* src = reinterpret_cast<const f4*>(a.h_in + srow * C + g * KS);
#pragma unroll
          for (int q = 0; q < KSP / 4; ++q) gb[c].v[q] = src[q];
        }
      }
    };
    auto load_w = [&](int k, f4 (&wv)[NCB][KSP / 4]) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        const f4* wp = reinterpret_cast<const f4*>(s_w + ((k * NCB + cb) * 64 + lane) * KSP);
#pragma unroll
        for (int q = 0; q < KSP / 4; ++q) wv[cb][q] = wp[q];
      }
    };
    auto mma_bf = [&](const int (&ks)[PCH], const G (&gb)[PCH]) {
      if constexpr (BF) {
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        if (ks[c] < 0) break;
        enter(ks[c]);
        uint4 wa[NCB][2];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const uint4* wp = reinterpret_cast<const uint4*>(s_w) + ((ks[c] * NCB + cb) * 64 + lane) * 2;
          wa[cb][0] = wp[0];
          wa[cb][1] = wp[1];
        }
        uint4 bh, bl;
        if constexpr (FIRST) {
          // 11 input bits: lane group 0 carries bits 0..7, group 1 bits 8..10
          // (exact in bf16), groups 2-3 zeros; products hi*x + lo*x
          const uint32_t bits = g < 2 ? (gb[c].word >> (8 * g)) & (g == 0 ? 0xFFu : 0x7u) : 0u;
          uint32_t wd[4];
#pragma unroll
          for (int pr = 0; pr < 4; ++pr)
            wd[pr] = (((bits >> (2 * pr)) & 1u) ? 0x3F80u : 0u) | (((bits >> (2 * pr + 1)) & 1u) ? 0x3F800000u : 0u);
          bh = make_uint4(wd[0], wd[1], wd[2], wd[3]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma_bf(wa[cb][0], bh, acc[cb]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma_bf(wa[cb][1], bh, acc[cb]);
        } else {
          bh = gb[c].hi;
          bl = gb[c].lo;
          // the three products, column blocks interleaved
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma_bf(wa[cb][0], bh, acc[cb]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma_bf(wa[cb][0], bl, acc[cb]);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma_bf(wa[cb][1], bh, acc[cb]);
        }
      }
      }
    };
    auto mma_f32 = [&](const int (&ks)[PCH], const G (&gb)[PCH]) {
      if constexpr (!BF) {
#pragma unroll
      for (int c = 0; c < PCH; ++c) {
        if (ks[c] < 0) break;
        enter(ks[c]);
        f4 wv[NCB][KSP / 4];
        load_w(ks[c], wv);
        float bsrc[KSP];
        if constexpr (FIRST) {
#pragma unroll
          for (int s = 0; s < KSP; ++s) bsrc[s] = (float)((gb[c].word >> (g * KS + s)) & 1u);
          // slot s = KS (padding) meets zero weights
        } else if constexpr (!BF) {
#pragma unroll
          for (int q = 0; q < KSP / 4; ++q)
#pragma unroll
            for (int e = 0; e < 4; ++e) bsrc[4 * q + e] = gb[c].v[q][e];
        }
        // column blocks interleaved: NCB independent accumulator chains
#pragma unroll
        for (int s = 0; s < KS; ++s)
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma4(wv[cb][s / 4][s % 4], bsrc[s], acc[cb]);
      }
      }
    };
    auto mma = [&](const int (&ks)[PCH], const G (&gb)[PCH]) {
      if constexpr (BF) mma_bf(ks, gb);
      else mma_f32(ks, gb);
    };
    {
      int ksA[PCH], ksB[PCH];
      G gA[PCH], gB[PCH];
      take(ksA);
      gather(ksA, gA);
      if constexpr (FIRST) {
        // fully unrolled (at most 27 offsets): straight-line code keeps the
        // compiler's wait counts exact across the pipeline's stages
        constexpr int ROUNDS = (27 + 2 * PCH - 1) / (2 * PCH);
#pragma unroll
        for (int it = 0; it < ROUNDS; ++it) {
          take(ksB);
          gather(ksB, gB);
          mma(ksA, gA);
          if (ksB[0] < 0) break;
          take(ksA);
          gather(ksA, gA);
          mma(ksB, gB);
          if (ksA[0] < 0) break;
        }
      } else {
        while (true) {
          take(ksB);
          gather(ksB, gB);
          mma(ksA, gA);
          if (ksB[0] < 0) break;
          take(ksA);
          gather(ksA, gA);
          mma(ksB, gB);
          if (ksA[0] < 0) break;
        }
      }
    }
    if (grp < 0) {
      while (gcur < 4) fold();  // every group folded, also the empty ones
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) out[cb] = tsum[cb];
    } else {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) out[cb] = acc[cb];
    }
    tr.b = b;
    tr.mo = mo;
    tr.prow = prow;
    tr.lvb = lvb;
    tr.valid = valid;
  };
  // Residual, ReLU, the children's X_B rows (full predictor) and the output row.
  auto epilogue = [&](const TileRef& tr, f4 (&acc)[NCB]) {
    const int b = tr.b;
    const int64_t mo = tr.mo, prow = tr.prow, lvb = tr.lvb;
    const bool valid = tr.valid;
    if (a.res) {  // residual block: ReLU(x + conv(.)), x read at the voxel's own row
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[cb] += *reinterpret_cast<const f4*>(a.res + prow * C + 16 * cb + 4 * g);
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[cb][e] = fmaxf(acc[cb][e], 0.0f);
    if (a.xb && valid) {  // children v of this voxel u: X_B[v] = F[u] + Emb_D[delta(v)]
      int64_t cmo = a.moff[b + 1];
      const int64_t cn = a.count[b + 1];
      const uint32_t code = a.code[lvb + (prow - mo)];
      const int64_t first = a.fc[lvb + (prow - mo)];
      if (cmo + cn > a.cap_model) cmo = -1;  // overflow (latched where the size was made): no writes
      int rank = 0;
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        if (cmo >= 0 && ((code >> d) & 1u)) {
          float* dst = a.xb + (cmo + first + rank) * C;
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb)
            *reinterpret_cast<f4*>(dst + 16 * cb + 4 * g) =
                acc[cb] + *reinterpret_cast<const f4*>(a.emb_d + d * C + 16 * cb + 4 * g);
          ++rank;
        }
      }
    }
    if (valid && a.h_out) {
      if constexpr (BF && !LAST) {
        // next layer's input as [hi plane | lo plane] of bf16 (split once per voxel)
        uint16_t* row = reinterpret_cast<uint16_t*>(a.h_out + prow * C);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          uint32_t h0, l0, h1, l1;
          split2(acc[cb][0], acc[cb][1], h0, l0);
          split2(acc[cb][2], acc[cb][3], h1, l1);
          *reinterpret_cast<uint2*>(row + 16 * cb + 4 * g) = make_uint2(h0, h1);
          *reinterpret_cast<uint2*>(row + C + 16 * cb + 4 * g) = make_uint2(l0, l1);
        }
      } else {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
          *reinterpret_cast<f4*>(a.h_out + prow * C + 16 * cb + 4 * g) = acc[cb];
      }
    }

  };

  if (!quads) {
    // Tile order (conv_tile): every XCD gets chunks from the whole tile range,
    // a sample of every scale of the launch, so the XCDs carry about the same
    // mix of cheap and expensive tiles (coarse scales have far more occupied
    // offsets per tile).  Inside a block the waves take the block's tiles
    // dynamically from an LDS counter: the first CONV_WAVES slots statically,
    // the rest first come, first served.
    for (int64_t slot = w;;) {
      const int64_t tile = conv_tile(slot, tch);
      if (tile >= total_tiles) break;
      TileRef tr;
      f4 acc[NCB];
      conv_sum(tile, -1, tr, acc);
      epilogue(tr, acc);
      if constexpr (LAST) head_epilogue<C, TWO, BF>(a, acc, s_h, lane, g, tr.valid, tr.prow, tr.mo, tr.lvb, s_mo[0]);
      int nxt = 0;
      if (lane == 0) nxt = atomicAdd(&s_next, 1);
      slot = CONV_WAVES + __builtin_amdgcn_readfirstlane(__shfl(nxt, 0));
    }
    return;
  }

  // Small launch (at most one tile per quad of waves): quad q of block x takes
  // tile x + q G, its wave i the offsets of group i, so a tile's serial MFMA
  // chain is split four ways.  The group sums meet in the weight area of LDS
  // (free once every conv loop is done) and are folded by wave 0 in the same
  // order as above; the 256-way head is split by symbol group the same way.
  // Every wave passes every barrier (no early exit below).
  {
    const int q = w >> 2, gi = w & 3;
    const int64_t tile = (int64_t)blockIdx.x + (int64_t)gridDim.x * q;
    const bool has = tile < total_tiles;  // wave-uniform
    TileRef tr{};
    f4 acc[NCB];
    if (has) conv_sum(tile, gi, tr, acc);
    __syncthreads();  // every conv loop of the block is done: the weight area is free
    f4* s_x = reinterpret_cast<f4*>(s_w);  // [quad][slot 0..3][NCB][64]: group sums 1-3, h
    float2* s_x2 = reinterpret_cast<float2*>(s_x + 16 * NCB * 64);  // [quad][group][64]: (gm, part)
    auto xs = [&](int slot, int cb) -> f4* { return s_x + ((q * 4 + slot) * NCB + cb) * 64 + lane; };
    if (has && gi > 0) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) *xs(gi - 1, cb) = acc[cb];
    }
    __syncthreads();
    if (has && gi == 0) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        f4 t = *reinterpret_cast<const f4*>(a.bias + 16 * cb + 4 * g);
        t += acc[cb];
        t += *xs(0, cb);
        t += *xs(1, cb);
        t += *xs(2, cb);
        acc[cb] = t;
      }
      epilogue(tr, acc);
      if constexpr (LAST && !TWO) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) *xs(3, cb) = acc[cb];  // h for the quad's other waves
      }
      if constexpr (LAST && TWO) head_epilogue<C, TWO, BF>(a, acc, s_h, lane, g, tr.valid, tr.prow, tr.mo, tr.lvb, s_mo[0]);
    }
    if constexpr (LAST && !TWO) {
      __syncthreads();
      if (has) {
        f4 h[NCB];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) h[cb] = *xs(3, cb);
        float gm, part;
        head_group<C, BF>(a, h, s_h, a.hb, lane, g, tr.valid, tr.prow, s_mo[0], gi, gm, part);
        s_x2[(q * 4 + gi) * 64 + lane] = make_float2(gm, part);
      }
      __syncthreads();
      if (has && gi == 0) {
        float m = -INFINITY, ssum = 0.0f;
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const float2 v = s_x2[(q * 4 + k) * 64 + lane];
          lse_merge(m, ssum, v.x, v.y);
        }
        lse_finish(a, m, ssum, g, tr.valid, tr.prow);
      }
    }
  }
}

// Tile order for the layers after the first: inside each window of TO_W
// consecutive voxels of a scale, voxels are grouped by an 11-bit signature of
// their neighbour occupancy (the 9 offsets of their own z plane and the two
// z faces), so a 16-voxel tile gathers voxels with similar neighbourhoods and
// the union of occupied offsets a tile must issue shrinks (14-bit scan: about
// 2.4x -> 1.6x the occupied pairs).  A voxel's result does not depend on which
// voxels share its tile (absent offsets add exact zeros), so any order, even
// the arrival order inside a group, gives the same outputs.  One block per
// window: counting sort in LDS.
constexpr int TO_W = 2048;
constexpr int TO_THREADS = 1024;
constexpr int TO_KEYS = 2048;

__global__ void __launch_bounds__(TO_THREADS) k_tile_order(int b_lo, int nsc, RowMap rm, int ks,
                                                           const int32_t* __restrict__ nbr, int32_t* __restrict__ perm) {
  __shared__ uint32_t s_cnt[TO_KEYS];
  __shared__ uint32_t s_wsum[TO_THREADS / 64];
  __shared__ int64_t s_n[NLEV], s_mo[NLEV];
  __shared__ int64_t s_w0, s_wmo, s_wn;
  const int tid = threadIdx.x;
  if (tid < nsc) {  // sizes of the launch's scales, loaded in parallel
    int64_t mo, n;
    scale_span(rm, b_lo + tid, mo, n);
    s_n[tid] = n;
    s_mo[tid] = mo;
  }
  for (int k = tid; k < TO_KEYS; k += TO_THREADS) s_cnt[k] = 0u;
  __syncthreads();
  if (tid == 0) {  // window blockIdx.x -> (scale, first voxel of the window)
    int64_t wacc = 0, w0 = -1;
    for (int i = 0; i < nsc; ++i) {
      const int64_t nw = (s_n[i] + TO_W - 1) / TO_W;
      if (w0 < 0 && (int64_t)blockIdx.x < wacc + nw) {
        w0 = ((int64_t)blockIdx.x - wacc) * TO_W;
        s_wmo = s_mo[i];
        s_wn = s_n[i];
      }
      wacc += nw;
    }
    s_w0 = w0;
  }
  __syncthreads();
  const int64_t w0 = s_w0;
  if (w0 < 0) return;  // beyond the last window (uniform over the block)
  const int64_t mo = s_wmo, n = s_wn;
  constexpr int PER = TO_W / TO_THREADS;
  uint32_t key[PER], rank[PER];
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int64_t i = w0 + e * TO_THREADS + tid;
    key[e] = TO_KEYS;  // absent
    if (i < n && ks == 3) {
      const int32_t* r = nbr + (mo + i) * NBR_STRIDE;
      const int4 a = *reinterpret_cast<const int4*>(r + 8), c = *reinterpret_cast<const int4*>(r + 12);
      const int4 d = *reinterpret_cast<const int4*>(r + 16);
      const int f4v = r[4], f22 = r[22];
      // offsets 9..17 (dz = 0), then 4 (dz = -1 face) and 22 (dz = +1 face)
      key[e] = (uint32_t)(a.y >= 0) | ((uint32_t)(a.z >= 0) << 1) | ((uint32_t)(a.w >= 0) << 2) |
               ((uint32_t)(c.x >= 0) << 3) | ((uint32_t)(c.y >= 0) << 4) | ((uint32_t)(c.z >= 0) << 5) |
               ((uint32_t)(c.w >= 0) << 6) | ((uint32_t)(d.x >= 0) << 7) | ((uint32_t)(d.y >= 0) << 8) |
               ((uint32_t)(f4v >= 0) << 9) | ((uint32_t)(f22 >= 0) << 10);
      rank[e] = atomicAdd(&s_cnt[key[e]], 1u);
    } else if (i < n) {
      // 5x5x5 map (stride 128): the same cells, k = (dx+2) + 5(dy+2) + 25(dz+2)
      const int32_t* r = nbr + (mo + i) * 128;
      const int32_t v[11] = {r[56], r[57], r[58], r[61], r[62], r[63], r[66], r[67], r[68], r[37], r[87]};
      uint32_t kk = 0;
#pragma unroll
      for (int j = 0; j < 11; ++j) kk |= (uint32_t)(v[j] >= 0) << j;
      key[e] = kk;
      rank[e] = atomicAdd(&s_cnt[key[e]], 1u);
    }
  }
  __syncthreads();
  // exclusive scan of the TO_KEYS counts: two per thread, wave scans, wave totals
  constexpr int KPT = TO_KEYS / TO_THREADS;
  uint32_t v[KPT], sum = 0;
#pragma unroll
  for (int e = 0; e < KPT; ++e) {
    v[e] = s_cnt[tid * KPT + e];
    sum += v[e];
  }
  uint32_t inc = sum;
  const int lane = tid & 63, w = tid >> 6;
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t t = (uint32_t)__shfl_up((int)inc, d);
    if (lane >= d) inc += t;
  }
  if (lane == 63) s_wsum[w] = inc;
  __syncthreads();
  uint32_t wbase = 0;
  for (int k = 0; k < w; ++k) wbase += s_wsum[k];
  uint32_t ex = wbase + inc - sum;
#pragma unroll
  for (int e = 0; e < KPT; ++e) {
    s_cnt[tid * KPT + e] = ex;
    ex += v[e];
  }
  __syncthreads();
#pragma unroll
  for (int e = 0; e < PER; ++e) {
    const int64_t i = w0 + e * TO_THREADS + tid;
    if (i < n) perm[mo + w0 + s_cnt[key[e]] + rank[e]] = (int32_t)(mo + i);
  }
}

// ---------------------------------------------------------------------------
// Inputs of the full predictor (Sec. 3.2): the neighbour maps of the scales
// it convolves on and the occupancy embeddings X_A = Emb_O[O^{d-1}] (Eq. 6),
// in one launch; one wave per tile of 16 voxels of the scales lo ..
// lo + nsc - 1, the first n_embed of which also get X_A rows.

// Last index si with pre[si] <= e (pre non-decreasing, 32 entries, pre[0] = 0
// <= e): binary lifting, si + step never exceeds 31.
__device__ __forceinline__ int scale_of(const int64_t* pre, int64_t e) {
  int si = 0;
#pragma unroll
  for (int step = 16; step; step >>= 1)
    if (pre[si + step] <= e) si += step;
  return si;
}

// Neighbour rows of a voxel of the base scale, whose parent scale is not
// stored: the 8 cells of lane group g located among the scale's n sorted
// Morton keys by 8 interleaved searches for the last key <= the cell
// (wave-uniform trip count; every probe stays below n).
__device__ __forceinline__ void base_cell_rows(uint64_t kf, int b, int g, const uint64_t* __restrict__ keys,
                                               int64_t n, int32_t (&nb)[8]) {
  const uint64_t key = morton_part(kf, b), fr = kf ^ key;  // frame id bits, in place
  const int x = (int)compact3(key), y = (int)compact3(key >> 1), z = (int)compact3(key >> 2);
  const int lim = 1 << b;
  uint64_t want[8];
  bool ok[8];
  int64_t at[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int k = 8 * g + j;
    const int ux = x + (k % 3) - 1, uy = y + (k / 3) % 3 - 1, uz = z + (k / 9) % 3 - 1;
    ok[j] = k < 27 && ux >= 0 && uy >= 0 && uz >= 0 && ux < lim && uy < lim && uz < lim;
    want[j] = ok[j] ? (fr | morton3((uint32_t)ux, (uint32_t)uy, (uint32_t)uz)) : 0ull;
    at[j] = 0;
  }
  for (int64_t len = n; len > 1;) {
    const int64_t half = len >> 1;
#pragma unroll
    for (int j = 0; j < 8; ++j) at[j] += (keys[at[j] + half] <= want[j]) ? half : 0;
    len -= half;
  }
#pragma unroll
  for (int j = 0; j < 8; ++j) nb[j] = (ok[j] && keys[at[j]] == want[j]) ? (int32_t)at[j] : -1;
}

template <int C>
__global__ void __launch_bounds__(256) k_top_prep(int lo, int nsc, int n_embed, int b0, RowMap rm,
                                                  const uint64_t* __restrict__ lv_key,
                                                  const uint8_t* __restrict__ lv_code, int64_t cap_pts,
                                                  const HashSlot* __restrict__ hash, int hash_lg,
                                                  const uint64_t* __restrict__ hreg, int fb,
                                                  const float* __restrict__ emb_o, int32_t* __restrict__ nbr,
                                                  float* __restrict__ X) {
  constexpr int Q = C / 16;  // f4 per lane of a row
  __shared__ uint64_t s_par[4][16][9];  // rows padded: the 16 voxels' cells in different banks
  __shared__ int64_t s_n[32], s_mo[32], s_tpre[32];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  if (tid < nsc) {  // sizes of the launch's scales, loaded in parallel
    int64_t o, n;
    scale_span(rm, lo + tid, o, n);
    s_n[tid] = n;
    s_mo[tid] = o;
  }
  __syncthreads();
  if (tid == 0) {
    int64_t acc = 0;
    for (int i = 0; i < nsc; ++i) {
      s_tpre[i] = acc;
      acc += (s_n[i] + 15) / 16;
    }
    for (int i = nsc; i < 32; ++i) s_tpre[i] = acc;
  }
  __syncthreads();
  const int64_t total = s_tpre[31];
  for (int64_t tile = (int64_t)blockIdx.x * 4 + w; tile < total; tile += (int64_t)gridDim.x * 4) {
    const int si = scale_of(s_tpre, tile);
    const int b = lo + si;
    const int64_t n = s_n[si], mo = s_mo[si];
    const int64_t row = (tile - s_tpre[si]) * 16 + r;
    const bool valid = row < n;
    const int64_t vr = valid ? row : n - 1;  // idle lanes search a real voxel
    const int64_t lvb = (int64_t)(b - b0) * cap_pts;
    int32_t nb[8];
    if (b == rm.b_ext)
      base_cell_rows(lv_key[lvb + vr], b, g, lv_key + lvb, n, nb);
    else
      parent_cell_rows(lv_key[lvb + vr], b, g, hash, hash_lg, hreg, fb, s_par[w][r], nb);
    if (valid) {
      int4* dst = reinterpret_cast<int4*>(nbr + (mo + vr) * NBR_STRIDE + 8 * g);
      dst[0] = make_int4(nb[0], nb[1], nb[2], nb[3]);
      dst[1] = make_int4(nb[4], nb[5], nb[6], nb[7]);
      if (si < n_embed) {
        const f4* e = reinterpret_cast<const f4*>(emb_o + (int)lv_code[lvb + vr] * C) + g * Q;
        f4* xr = reinterpret_cast<f4*>(X + (mo + vr) * C) + g * Q;
#pragma unroll
        for (int q = 0; q < Q; ++q) xr[q] = e[q];
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Large kernels and wide layers of the full predictor (5x5x5 kernels, C up to
// 128: the paper's large variant is c128, k5).

// Neighbour rows of a voxel for a 5x5x5 kernel.  The 125 cells around v span
// x-2 .. x+2 on each axis, i.e. the parents p-1 .. p+1: 27 cells of the
// parent scale.  Lane (r, g) probes parent cells e = g, g+4, ... (e = (ex+1) +
// 3(ey+1) + 9(ez+1)), the hits are exchanged through par (27 LDS slots of
// voxel r), and the lane ends with the rows of offsets k = 32g .. 32g+31,
// k = (dx+2) + 5(dy+2) + 25(dz+2) (125 .. 127 padding; -1: absent or
// off-grid).
__device__ __forceinline__ void parent_cell_rows5(uint64_t kf, int b, int g, const HashSlot* __restrict__ hash,
                                                  int hash_lg, const uint64_t* __restrict__ hreg, int fb,
                                                  volatile uint64_t* par, int32_t (&nb)[32]) {
  const uint64_t key = morton_part(kf, b), fr = frame_part(kf, b) << (3 * (b - 1));
  const int x = (int)compact3(key), y = (int)compact3(key >> 1), z = (int)compact3(key >> 2);
  const int px = x >> 1, py = y >> 1, pz = z >> 1;
  const int plim = 1 << (b - 1);
  uint64_t tk[7];
#pragma unroll
  for (int i = 0; i < 7; ++i) {
    const int e = g + 4 * i;
    const int cx = px + e % 3 - 1, cy = py + (e / 3) % 3 - 1, cz = pz + e / 9 - 1;
    tk[i] = (e < 27 && cx >= 0 && cy >= 0 && cz >= 0 && cx < plim && cy < plim && cz < plim)
                ? tag_key(fr | morton3((uint32_t)cx, (uint32_t)cy, (uint32_t)cz), b - 1, fb)
                : 0ull;
  }
  uint2 hit[7];
  hash_find_n<7>(hash, hash_lg, hash_region(hreg, hash_lg, frame_part(kf, b)), tk, hit);
#pragma unroll
  for (int i = 0; i < 7; ++i)
    if (g + 4 * i < 27) par[g + 4 * i] = ((uint64_t)hit[i].y << 32) | hit[i].x;
  __builtin_amdgcn_wave_barrier();
  const int lim = 1 << b;
#pragma unroll
  for (int j = 0; j < 32; ++j) {
    const int k = 32 * g + j;
    const int ux = x + k % 5 - 2, uy = y + (k / 5) % 5 - 2, uz = z + k / 25 - 2;
    nb[j] = -1;
    if (k < 125 && ux >= 0 && uy >= 0 && uz >= 0 && ux < lim && uy < lim && uz < lim) {
      const int e = ((ux >> 1) - px + 1) + 3 * ((uy >> 1) - py + 1) + 9 * ((uz >> 1) - pz + 1);
      const uint64_t pc = par[e];
      const uint32_t first = (uint32_t)pc, code = (uint32_t)(pc >> 32);
      const uint32_t d = (uint32_t)((ux & 1) | ((uy & 1) << 1) | ((uz & 1) << 2));
      if ((code >> d) & 1u) nb[j] = (int32_t)first + __popc(code & ((1u << d) - 1u));
    }
  }
}

// Base-scale rows for a 5x5x5 kernel: the searches of base_cell_rows, eight
// interleaved at a time over the 32 entries of the lane.
__device__ __forceinline__ void base_cell_rows5(uint64_t kf, int b, int g, const uint64_t* __restrict__ keys,
                                                int64_t n, int32_t (&nb)[32]) {
  const uint64_t key = morton_part(kf, b), fr = kf ^ key;
  const int x = (int)compact3(key), y = (int)compact3(key >> 1), z = (int)compact3(key >> 2);
  const int lim = 1 << b;
#pragma unroll
  for (int j0 = 0; j0 < 32; j0 += 8) {
    uint64_t want[8];
    bool ok[8];
    int64_t at[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = 32 * g + j0 + j;
      const int ux = x + k % 5 - 2, uy = y + (k / 5) % 5 - 2, uz = z + k / 25 - 2;
      ok[j] = k < 125 && ux >= 0 && uy >= 0 && uz >= 0 && ux < lim && uy < lim && uz < lim;
      want[j] = ok[j] ? (fr | morton3((uint32_t)ux, (uint32_t)uy, (uint32_t)uz)) : 0ull;
      at[j] = 0;
    }
    for (int64_t len = n; len > 1;) {
      const int64_t half = len >> 1;
#pragma unroll
      for (int j = 0; j < 8; ++j) at[j] += (keys[at[j] + half] <= want[j]) ? half : 0;
      len -= half;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) nb[j0 + j] = (ok[j] && keys[at[j]] == want[j]) ? (int32_t)at[j] : -1;
  }
}

// k_top_prep for a 5x5x5 kernel: neighbour maps of stride 128 and X_A rows.
template <int C>
__global__ void __launch_bounds__(256) k_top_prep5(int lo, int nsc, int n_embed, int b0, RowMap rm,
                                                   const uint64_t* __restrict__ lv_key,
                                                   const uint8_t* __restrict__ lv_code, int64_t cap_pts,
                                                   const HashSlot* __restrict__ hash, int hash_lg,
                                                  const uint64_t* __restrict__ hreg, int fb,
                                                   const float* __restrict__ emb_o, int32_t* __restrict__ nbr,
                                                   float* __restrict__ X) {
  constexpr int Q = C / 16;
  __shared__ uint64_t s_par[4][16][27];
  __shared__ int64_t s_n[32], s_mo[32], s_tpre[32];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  if (tid < nsc) {
    int64_t o, n;
    scale_span(rm, lo + tid, o, n);
    s_n[tid] = n;
    s_mo[tid] = o;
  }
  __syncthreads();
  if (tid == 0) {
    int64_t acc = 0;
    for (int i = 0; i < nsc; ++i) {
      s_tpre[i] = acc;
      acc += (s_n[i] + 15) / 16;
    }
    for (int i = nsc; i < 32; ++i) s_tpre[i] = acc;
  }
  __syncthreads();
  const int64_t total = s_tpre[31];
  for (int64_t tile = (int64_t)blockIdx.x * 4 + w; tile < total; tile += (int64_t)gridDim.x * 4) {
    const int si = scale_of(s_tpre, tile);
    const int b = lo + si;
    const int64_t n = s_n[si], mo = s_mo[si];
    const int64_t row = (tile - s_tpre[si]) * 16 + r;
    const bool valid = row < n;
    const int64_t vr = valid ? row : n - 1;
    const int64_t lvb = (int64_t)(b - b0) * cap_pts;
    int32_t nb[32];
    if (b == rm.b_ext)
      base_cell_rows5(lv_key[lvb + vr], b, g, lv_key + lvb, n, nb);
    else
      parent_cell_rows5(lv_key[lvb + vr], b, g, hash, hash_lg, hreg, fb, s_par[w][r], nb);
    if (valid) {
      int4* dst = reinterpret_cast<int4*>(nbr + (mo + vr) * 128 + 32 * g);
#pragma unroll
      for (int q = 0; q < 8; ++q) dst[q] = make_int4(nb[4 * q], nb[4 * q + 1], nb[4 * q + 2], nb[4 * q + 3]);
      if (si < n_embed) {
        const f4* e = reinterpret_cast<const f4*>(emb_o + (int)lv_code[lvb + vr] * C) + g * Q;
        f4* xr = reinterpret_cast<f4*>(X + (mo + vr) * C) + g * Q;
#pragma unroll
        for (int q = 0; q < Q; ++q) xr[q] = e[q];
      }
    }
  }
}

// Offset set of up to 128 offsets (wave-uniform).
struct OffMask {
  uint64_t lo = 0, hi = 0;
  __device__ __forceinline__ void set(int o) {
    if (o < 64) lo |= 1ull << o;
    else hi |= 1ull << (o - 64);
  }
  // lowest offset, removed from the set (-1 when empty)
  __device__ __forceinline__ int pop() {
    if (lo) {
      const int k = __builtin_ctzll(lo);
      lo &= lo - 1ull;
      return k;
    }
    if (hi) {
      const int k = 64 + __builtin_ctzll(hi);
      hi &= hi - 1ull;
      return k;
    }
    return -1;
  }
};

constexpr int CW_THREADS = 512;
constexpr int CW_SPLIT_ROUNDS = 2;  // column split while a block has at most this many tile sets
constexpr int CW_WAVES = CW_THREADS / 64;

// Sparse conv C -> C (ReLU, optional residual input, child scatter and row
// store as in k_conv) with the weights streamed through LDS, for layers whose
// weights do not fit in it (a 5x5x5 kernel at C = 128 holds 8 MB).  A block
// takes groups of CW_WAVES tiles, one per wave.  For each offset in the union
// of the group's occupied offsets, in ascending order, the block stages that
// offset's C x C weights in LDS (double buffered: the next offset's loads are
// issued before the current MFMAs), and each wave whose tile has the offset
// accumulates its gathered neighbour rows on fp32 MFMA 16x16x4 in the layout
// of k_conv; the wave's next gather is issued before its MFMAs.  A voxel sums
// its offsets in ascending order whatever its group, so results do not depend
// on the grouping.
template <int C, int KV>
__global__ void __launch_bounds__(CW_THREADS) k_convw(ConvArgs a) {
  constexpr int NCB = C / 16;
  constexpr int KS = C / 4;  // input channels of a lane group (one contiguous slice of a row)
  constexpr int NBS = KV > 27 ? 128 : NBR_STRIDE;
  constexpr int EPL = NBS / 4;  // map entries per lane
  constexpr int WQ = C * C / 4;  // 16-byte words of one offset's packed weights
  __shared__ __attribute__((aligned(16))) float s_w[2][C * C];
  __shared__ uint64_t s_mask[CW_WAVES][2];
  __shared__ int64_t s_tpre[NLEV + 1];
  __shared__ int64_t s_nv[NLEV];
  __shared__ int64_t s_mo[NLEV];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  const int nsc = a.b_hi - a.b_lo + 1;
  const RowMap rm{a.count, a.moff, a.cap_model, a.b_ext, a.ext_off, a.cap_rows};
  int64_t total_tiles = 0;
  for (int i = 0; i < nsc; ++i) {
    int64_t mo, nb;
    scale_span(rm, a.b_lo + i, mo, nb);
    total_tiles += (nb + 15) / 16;
  }
  const int64_t groups = (total_tiles + CW_WAVES - 1) / CW_WAVES;
  const int64_t tch = groups / 64 < 4 ? 4 : (groups / 64 > 64 ? 64 : groups / 64);
  // Column split for launches with few tiles: a block takes TPB tiles and
  // wave w computes column block w % NCB of tile w / NCB, so a tile's serial
  // walk over its offsets is spread over NCB waves (each output channel's
  // MFMA chain is the same as with one wave per tile) and the block walks the
  // union of TPB tiles instead of CW_WAVES.
  constexpr int TPB = CW_WAVES / NCB;
  const int64_t sets = (total_tiles + TPB - 1) / TPB;
  const bool split = NCB > 1 && sets <= (int64_t)gridDim.x * CW_SPLIT_ROUNDS;  // uniform
  const int64_t nwork = split ? sets : groups;
  if (split ? (int64_t)blockIdx.x >= sets : conv_tile(0, tch) >= groups) return;  // whole block idle
  if (tid == 0) {
    int64_t acc = 0;
    for (int i = 0; i < nsc; ++i) {
      int64_t mo, nb;
      scale_span(rm, a.b_lo + i, mo, nb);
      s_tpre[i] = acc;
      s_nv[i] = nb;
      s_mo[i] = mo;
      acc += (nb + 15) / 16;
    }
    for (int i = nsc; i <= NLEV; ++i) s_tpre[i] = acc;
  }
  const f4* wsrc = reinterpret_cast<const f4*>(a.w);
  const int cb0 = split ? w % NCB : 0;  // the wave's (first) column block
  for (int64_t gs = 0;; ++gs) {
    const int64_t grp = split ? (int64_t)blockIdx.x + gs * (int64_t)gridDim.x : conv_tile(gs, tch);  // block-uniform
    if (grp >= nwork) break;
    __syncthreads();  // prefix visible; the previous group is done with s_mask and s_w
    const int64_t tile = split ? grp * TPB + w / NCB : grp * CW_WAVES + w;
    const bool have = tile < total_tiles;
    int b = a.b_lo;
    int64_t mo = 0, prow = 0, lvb = 0;
    bool valid = false;
    if (have) {
      int si = 0;
#pragma unroll
      for (int i = 1; i < NLEV; ++i) si += (s_tpre[i] <= tile) ? 1 : 0;
      b = a.b_lo + si;
      const int64_t nvox = s_nv[si];
      mo = s_mo[si];
      const int64_t row = (tile - s_tpre[si]) * 16 + r;
      valid = row < nvox;
      const int64_t pos = mo + (valid ? row : nvox - 1);  // idle lanes read a real row
      prow = a.perm ? (int64_t)a.perm[pos] : pos;          // with a tile order, slot -> row
      lvb = (int64_t)(b - a.b0) * a.cap_pts;
    }
    // occupied offsets of the wave's tile (wave-uniform), from the map rows
    OffMask own;
    {
      int32_t nbv[EPL];
#pragma unroll
      for (int q = 0; q < EPL / 4; ++q) {
        int4 t = make_int4(-1, -1, -1, -1);
        if (have) t = reinterpret_cast<const int4*>(a.nbr + prow * NBS + EPL * g)[q];
        nbv[4 * q] = t.x;
        nbv[4 * q + 1] = t.y;
        nbv[4 * q + 2] = t.z;
        nbv[4 * q + 3] = t.w;
      }
#pragma unroll
      for (int j = 0; j < EPL; ++j) {
        const uint64_t bal = __ballot(valid && nbv[j] >= 0);
#pragma unroll
        for (int gg = 0; gg < 4; ++gg)
          if ((bal >> (16 * gg)) & 0xFFFFull) own.set(gg * EPL + j);
      }
    }
    if (lane == 0) {
      s_mask[w][0] = own.lo;
      s_mask[w][1] = own.hi;
    }
    __syncthreads();
    OffMask uni;
    for (int ww = 0; ww < CW_WAVES; ++ww) {
      uni.lo |= s_mask[ww][0];
      uni.hi |= s_mask[ww][1];
    }
    // each lane reads its own voxel's map entry of an offset two of the
    // wave's offsets ahead of its use, and gathers one offset ahead
    const int32_t* maprow = a.nbr + prow * NBS;
    auto entry = [&](int k) -> int32_t { return (k >= 0 && have) ? maprow[k] : -1; };
    auto gather = [&](int32_t nn, f4 (&x)[KS / 4]) {
      const int64_t srow = (valid && nn >= 0) ? mo + nn : a.cap_model;  // absent: the zero row
      const f4* src = reinterpret_cast<const f4*>(a.h_in + srow * C + g * KS);
#pragma unroll
      for (int q = 0; q < KS / 4; ++q) x[q] = src[q];
    };
    // acc[j] holds column block cb0 + j (split: j = 0 only)
    f4 acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[cb] = *reinterpret_cast<const f4*>(a.bias + 16 * (cb0 + (split ? 0 : cb)) + 4 * g);
    f4 xa[KS / 4], xb[KS / 4];
    int ko = own.pop();
    const int32_t eo = entry(ko);
    int kq = own.pop();
    int32_t eq = entry(kq);
    if (ko >= 0) gather(eo, xa);
    int kc = uni.pop();
    Staged<WQ, CW_THREADS> stw;
    if (kc >= 0) {  // always: wave 0 has a valid voxel, whose own centre is occupied
      stw.load(wsrc + (int64_t)kc * WQ, tid);
      stw.store(reinterpret_cast<f4*>(s_w[0]), tid);
    }
    __syncthreads();
    int buf = 0;
    while (kc >= 0) {  // block-uniform
      const int kn = uni.pop();
      if (kn >= 0) stw.load(wsrc + (int64_t)kn * WQ, tid);
      if (kc == ko) {
        const int kr = own.pop();
        const int32_t er = entry(kr);
        if (kq >= 0) gather(eq, xb);
        const float* wb = s_w[buf];
        if (split) {
#pragma unroll
          for (int q = 0; q < KS / 4; ++q) {
            const f4 wv = reinterpret_cast<const f4*>(wb)[(cb0 * (KS / 4) + q) * 64 + lane];
#pragma unroll
            for (int e = 0; e < 4; ++e) acc[0] = mfma4(wv[e], xa[q][e], acc[0]);
          }
        } else {
#pragma unroll
          for (int q = 0; q < KS / 4; ++q) {
            f4 wv[NCB];
#pragma unroll
            for (int cb = 0; cb < NCB; ++cb) wv[cb] = reinterpret_cast<const f4*>(wb)[(cb * (KS / 4) + q) * 64 + lane];
#pragma unroll
            for (int e = 0; e < 4; ++e)
#pragma unroll
              for (int cb = 0; cb < NCB; ++cb) acc[cb] = mfma4(wv[cb][e], xa[q][e], acc[cb]);
          }
        }
#pragma unroll
        for (int q = 0; q < KS / 4; ++q) xa[q] = xb[q];
        ko = kq;
        kq = kr;
        eq = er;
      }
    if (kn >= 0) stw.store(reinterpret_cast<f4*>(s_w[buf ^ 1]), tid);
      __syncthreads();
      buf ^= 1;
      kc = kn;
    }
    if (!have) continue;
    const int ncw = split ? 1 : NCB;  // column blocks this wave holds: cb0 .. cb0 + ncw - 1
    if (a.res) {  // residual block: ReLU(x + conv(.)), x read at the voxel's own row
#pragma unroll
      for (int j = 0; j < NCB; ++j)
        if (j < ncw) acc[j] += *reinterpret_cast<const f4*>(a.res + prow * C + 16 * (cb0 + j) + 4 * g);
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[cb][e] = fmaxf(acc[cb][e], 0.0f);
    if (a.xb && valid) {  // children v of this voxel u: X_B[v] = F[u] + Emb_D[delta(v)]
      int64_t cmo = a.moff[b + 1];
      const int64_t cn = a.count[b + 1];
      const uint32_t code = a.code[lvb + (prow - mo)];
      const int64_t first = a.fc[lvb + (prow - mo)];
      if (cmo + cn > a.cap_model) cmo = -1;  // overflow (latched where the size was made): no writes
      int rank = 0;
#pragma unroll
      for (int d = 0; d < 8; ++d) {
        if (cmo >= 0 && ((code >> d) & 1u)) {
          float* dst = a.xb + (cmo + first + rank) * C;
#pragma unroll
          for (int j = 0; j < NCB; ++j)
            if (j < ncw)
              *reinterpret_cast<f4*>(dst + 16 * (cb0 + j) + 4 * g) =
                  acc[j] + *reinterpret_cast<const f4*>(a.emb_d + d * C + 16 * (cb0 + j) + 4 * g);
          ++rank;
        }
      }
    }
    if (valid && a.h_out) {
#pragma unroll
      for (int j = 0; j < NCB; ++j)
        if (j < ncw) *reinterpret_cast<f4*>(a.h_out + prow * C + 16 * (cb0 + j) + 4 * g) = acc[j];
    }
  }
}

// The head on stored last-layer features h_in (rows of the scales b_lo ..
// b_hi), for layers computed by k_convw: one wave per tile of 16 voxels, the
// head weights in LDS, the same arithmetic as the fused head of k_conv.
// threads of a k_headw block: the two-stage head at C >= 64 needs more
// registers than 16 waves per CU allow
template <int C, bool TWO>
constexpr int headw_threads() { return (TWO && C >= 64) ? 256 : 1024; }

template <int C, bool TWO>
__global__ void __launch_bounds__((headw_threads<C, TWO>())) k_headw(ConvArgs a) {
  constexpr int NCB = C / 16;
  constexpr int HT = headw_threads<C, TWO>();
  constexpr int HWV = HT / 64;
  constexpr int HQ = (TWO ? 2 : 16) * 64 * (C / 4) / 4;  // 16-byte words of the packed head
  __shared__ __attribute__((aligned(16))) float s_h[HQ * 4];
  __shared__ int64_t s_tpre[NLEV + 1];
  __shared__ int64_t s_nv[NLEV];
  __shared__ int64_t s_mo[NLEV];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, r = lane & 15, g = lane >> 4;
  const int nsc = a.b_hi - a.b_lo + 1;
  const RowMap rm{a.count, a.moff, a.cap_model, -1, 0, a.cap_model + 1};
  Staged<HQ, HT> sth;
  sth.load(reinterpret_cast<const f4*>(a.hw), tid);
  if (tid == 0) {
    int64_t acc = 0;
    for (int i = 0; i < nsc; ++i) {
      int64_t mo, nb;
      scale_span(rm, a.b_lo + i, mo, nb);
      s_tpre[i] = acc;
      s_nv[i] = nb;
      s_mo[i] = mo;
      acc += (nb + 15) / 16;
    }
    for (int i = nsc; i <= NLEV; ++i) s_tpre[i] = acc;
  }
  sth.store(reinterpret_cast<f4*>(s_h), tid);
  __syncthreads();
  const int64_t total = s_tpre[NLEV];
  for (int64_t tile = (int64_t)blockIdx.x * HWV + w; tile < total; tile += (int64_t)gridDim.x * HWV) {
    int si = 0;
#pragma unroll
    for (int i = 1; i < NLEV; ++i) si += (s_tpre[i] <= tile) ? 1 : 0;
    const int b = a.b_lo + si;
    const int64_t nvox = s_nv[si], mo = s_mo[si];
    const int64_t row = (tile - s_tpre[si]) * 16 + r;
    const bool valid = row < nvox;
    const int64_t prow = mo + (valid ? row : nvox - 1);
    const int64_t lvb = (int64_t)(b - a.b0) * a.cap_pts;
    f4 acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[cb] = *reinterpret_cast<const f4*>(a.h_in + prow * C + 16 * cb + 4 * g);
    head_epilogue<C, TWO, false>(a, acc, s_h, lane, g, valid, prow, mo, lvb, s_mo[0]);
  }
}

template <int C, bool FIRST, bool LAST, bool TWO, bool BF>
hipError_t run_conv(Ctx& c, const ConvArgs& a) {
  // one block per CU stages the weights once for its 16 waves
  if (c.ext_start) {  // timed: the events are the dispatch's own start and end
    hipExtLaunchKernelGGL((k_conv<C, FIRST, LAST, TWO, BF>), dim3(256), dim3(CONV_THREADS), 0, c.stream,
                          c.ext_start, c.ext_stop, 0u, a);
    c.ext_start = c.ext_stop = nullptr;
  } else {
    hipLaunchKernelGGL((k_conv<C, FIRST, LAST, TWO, BF>), dim3(256), dim3(CONV_THREADS), 0, c.stream, a);
  }
  return hipGetLastError();
}

template <int C, bool BF>
hipError_t run_layer(Ctx& c, bool first, bool last, bool two, const ConvArgs& a) {
  if (first && last)
    return two ? run_conv<C, true, true, true, BF>(c, a) : run_conv<C, true, true, false, BF>(c, a);
  if (first) return run_conv<C, true, false, false, BF>(c, a);
  if (last) return two ? run_conv<C, false, true, true, BF>(c, a) : run_conv<C, false, true, false, BF>(c, a);
  return run_conv<C, false, false, false, BF>(c, a);
}

// Stage 2 of the two-stage head for one scale from the stored features of the
// last conv layer and a given S1 per voxel (decoder).  One wave per tile of
// 16 voxels, the same tile split and arithmetic as the fused path.
template <int C, bool BF>
__global__ void __launch_bounds__(256) k_head2(int b, const int32_t* __restrict__ count,
                                               const int32_t* __restrict__ moff, int64_t cap_model,
                                               const float* __restrict__ hL, const uint8_t* __restrict__ s1,
                                               const uint8_t* __restrict__ code, const float* __restrict__ hw2,
                                               const float* __restrict__ hb2, const float* __restrict__ emb,
                                               float* __restrict__ lse2, float* __restrict__ logits2,
                                               uint8_t* __restrict__ s1_out, uint32_t* err) {
  constexpr int NCB = C / 16;
  const int lane = threadIdx.x & 63, r = lane & 15, g = lane >> 4;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;  // overflow was latched where the size was made
  const int64_t ntiles = (n + 15) / 16;
  const int wpb = blockDim.x / 64;
  const f4* hp = reinterpret_cast<const f4*>(hw2) + lane * (C / 16);
  for (int64_t tile = (int64_t)blockIdx.x * wpb + (threadIdx.x >> 6); tile < ntiles;
       tile += (int64_t)gridDim.x * wpb) {
    const int64_t row = tile * 16 + r;
    const bool valid = row < n;
    const int64_t vr = valid ? row : n - 1;
    const int64_t prow = mo + vr;
    f4 h[NCB];
#pragma unroll
    for (int q = 0; q < NCB; ++q) h[q] = *reinterpret_cast<const f4*>(hL + prow * C + 16 * q + 4 * g);
    int a1 = s1 ? s1[vr] : (code[vr] & 15);
    if (a1 > 15) {
      if (valid) latch(err, ERR_SYMBOL);
      a1 = 0;
    }
    f4 h2[NCB];
    add_emb<C>(h, emb + a1 * C, g, h2);
    f4 z2;
    if constexpr (BF) {
      uint4 bh, bl;
      head_operand_bf<C>(h2, bh, bl);
      z2 = head16_bf<C>(reinterpret_cast<const uint4*>(hw2) + lane * 2, hb2, bh, bl, g);
    } else {
      z2 = head16<C>(hp, hb2, h2, g);
    }
    const float l2 = lse16(z2);
    if (valid && g == 0) {
      lse2[prow] = l2;
      s1_out[prow] = (uint8_t)a1;
    }
    if (valid && logits2) *reinterpret_cast<f4*>(logits2 + row * 16 + 4 * g) = z2;
  }
}

}  // namespace

hipError_t launch_pack_weights(Ctx& c, const reno_weights& w) {
  ProfScope ps_(c, RENO_K_OTHER);
  const int C = c.p.channels;
  int c_in = RENO_IN_FEATURES;
  const bool bf = c.p.precision == RENO_PREC_BF16X3;
  if (c.p.model_mode == RENO_MODEL_TOP) {  // four C -> C convs (fp32) and the two embeddings
    for (int l = 0; l < 4; ++l) {
      if (c.wide())
        hipLaunchKernelGGL(k_pack_conv_wide, dim3(1024), dim3(256), 0, c.stream, w.top_w[l], C, c.kvol(),
                           c.w_conv[l]);
      else
        hipLaunchKernelGGL(k_pack_conv, dim3(256), dim3(256), 0, c.stream, w.top_w[l], C, C, C / 4, C / 4,
                           c.kvol(), c.w_conv[l]);
      hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(256), 0, c.stream, w.top_b[l], c.w_bias[l], C);
    }
    hipLaunchKernelGGL(k_copy_f32, dim3(32), dim3(256), 0, c.stream, w.emb_o, c.w_embo, 256 * C);
    hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(256), 0, c.stream, w.emb_d, c.w_embd, 8 * C);
  }
  for (int l = 0; l < c.p.layers && c.p.model_mode != RENO_MODEL_TOP; ++l) {
    const int KS = (c_in + 3) / 4;
    const int KSP = (KS + 3) & ~3;
    if (bf)
      hipLaunchKernelGGL(k_pack_conv_bf, dim3(64), dim3(256), 0, c.stream, w.conv_w[l], c_in, C,
                         reinterpret_cast<uint32_t*>(c.w_conv[l]));
    else
      hipLaunchKernelGGL(k_pack_conv, dim3(64), dim3(256), 0, c.stream, w.conv_w[l], c_in, C, KS, KSP, 27,
                         c.w_conv[l]);
    hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(256), 0, c.stream, w.conv_b[l], c.w_bias[l], C);
    c_in = C;
  }
  if (c.p.head_mode == RENO_HEAD_TWO_STAGE) {
    // packed blocks [stage 1][stage 2], biases [b1 | b2], plain [C][H1 | H2]
    const int blk = bf ? 64 * 8 : 64 * (C / 4);
    if (bf) {
      uint32_t* hw = reinterpret_cast<uint32_t*>(c.w_head);
      hipLaunchKernelGGL(k_pack_head_bf, dim3(1), dim3(256), 0, c.stream, w.head1_w, C, 16, hw);
      hipLaunchKernelGGL(k_pack_head_bf, dim3(1), dim3(256), 0, c.stream, w.head2_w, C, 16, hw + blk);
    } else {
      hipLaunchKernelGGL(k_pack_head, dim3(4), dim3(256), 0, c.stream, w.head1_w, C, 16, c.w_head);
      hipLaunchKernelGGL(k_pack_head, dim3(4), dim3(256), 0, c.stream, w.head2_w, C, 16, c.w_head + blk);
    }
    hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(64), 0, c.stream, w.head1_b, c.w_hbias, 16);
    hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(64), 0, c.stream, w.head2_b, c.w_hbias + 16, 16);
    hipLaunchKernelGGL(k_put_cols16, dim3(2), dim3(256), 0, c.stream, w.head1_w, C, 0, c.w_head_plain);
    hipLaunchKernelGGL(k_put_cols16, dim3(2), dim3(256), 0, c.stream, w.head2_w, C, 16, c.w_head_plain);
    hipLaunchKernelGGL(k_copy_f32, dim3(2), dim3(256), 0, c.stream, w.emb_s1, c.w_emb, 16 * C);
    hipLaunchKernelGGL(k_transpose_head, dim3(2), dim3(256), 0, c.stream, w.head1_w, C, 16, 0, c.w_head_t);
    hipLaunchKernelGGL(k_transpose_head, dim3(2), dim3(256), 0, c.stream, w.head2_w, C, 16, 16, c.w_head_t);
  } else {
    if (bf)
      hipLaunchKernelGGL(k_pack_head_bf, dim3(16), dim3(256), 0, c.stream, w.head_w, C, 256,
                         reinterpret_cast<uint32_t*>(c.w_head));
    else
      hipLaunchKernelGGL(k_pack_head, dim3(32), dim3(256), 0, c.stream, w.head_w, C, 256, c.w_head);
    hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(256), 0, c.stream, w.head_b, c.w_hbias, 256);
    hipLaunchKernelGGL(k_copy_f32, dim3(32), dim3(256), 0, c.stream, w.head_w, c.w_head_plain,
                       C * 256);
    hipLaunchKernelGGL(k_transpose_head, dim3(32), dim3(256), 0, c.stream, w.head_w, C, 256, 0, c.w_head_t);
  }
  return hipGetLastError();
}

// Full predictor on the scales b_lo .. b_hi (Sec. 3.2, Eqs. 6-9):
//   neighbour maps of scales b_lo-1 .. b_hi, X_A = Emb_O[O^{d-1}] on scales
//   b_lo-1 .. b_hi-1 (h_c)                                        one prep launch
//   T = ReLU(conv_A1(X_A))                                        (h_b)
//   F_A = ReLU(X_A + conv_A2(T)), scattered to the children as
//   X_B = F_A[parent] + Emb_D[delta] on scales b_lo .. b_hi       (h_d; F_A itself is not stored)
//   T = ReLU(conv_B1(X_B))                                        (h_b)
//   F_B = ReLU(X_B + conv_B2(T)), fused with the head             (h_a)
// The base scale's rows live past the zero row.  F_B of earlier calls is
// never overwritten (code lengths of a scale stay valid after the next
// scale's call).
hipError_t launch_top(Ctx& c, int b_lo, int b_hi, float* logits, bool second) {
  const int b0 = c.b0();
  const int64_t ext_off = c.cap_model + 1;
  const RowMap rm{c.d_count, c.d_moff, (int64_t)c.cap_model, b0, ext_off, c.cap_rows()};
  const int C = c.p.channels;
  const int n_lo = b_lo - 1;  // stage A runs one scale below stage B
  {
    ProfScope ps_(c, RENO_K_TOP_INPUT);
    const int blocks = (int)std::min<int64_t>(2048, (c.cap_rows() + 63) / 64);
#define RENO_PREP(CC)                                                                                         \
  hipLaunchKernelGGL(k_top_prep<CC>, dim3(blocks), dim3(256), 0, c.stream, n_lo, b_hi - n_lo + 1, b_hi - n_lo, b0, \
                     rm, c.lv_key, c.lv_code, (int64_t)c.cap_pts, c.d_hash, c.hash_lg, c.hreg(), c.fbits, c.w_embo, \
                     c.d_nbr, c.h_c)
    if (C == 32) RENO_PREP(32); else RENO_PREP(16);
#undef RENO_PREP
  }
  ConvArgs a{};
  a.b0 = b0;
  a.count = c.d_count;
  a.moff = c.d_moff;
  a.cap_pts = c.cap_pts;
  a.cap_model = c.cap_model;
  a.lv_key = c.lv_key;
  a.lv_feat = c.lv_feat;
  a.hash = c.d_hash;
  a.hash_lg = c.hash_lg;
  a.hreg = c.hreg();
  a.fb = c.fbits;
  a.nbr = c.d_nbr;
  a.zero_feat = (int64_t)c.nlv * c.cap_pts;
  a.hb = c.w_hbias;
  a.hw = c.w_head;
  a.lse = c.d_lse;
  a.err = c.d_err;
  a.emb = c.w_emb;
  a.s1_code = second ? c.lv_code : nullptr;
  a.lse2 = c.d_lse2;
  a.s1_out = c.d_s1;
  a.b_ext = b0;
  a.ext_off = ext_off;
  a.cap_rows = c.cap_rows();
  a.emb_d = c.w_embd;
  a.code = c.lv_code;
  a.fc = c.lv_fc;
  const bool two = c.p.head_mode == RENO_HEAD_TWO_STAGE;
  if (b_lo != b_hi || b_lo >= c.B - 2) {  // sorted tiles, as for the plain model
    ProfScope pso_(c, RENO_K_OTHER);
    const int nsc = b_hi - n_lo + 1;
    const int64_t windows = (c.cap_model + c.cap_pts + TO_W - 1) / TO_W + nsc;
    hipLaunchKernelGGL(k_tile_order, dim3((unsigned)windows), dim3(TO_THREADS), 0, c.stream, n_lo, nsc, rm, 3,
                       c.d_nbr, c.d_perm);
    a.perm = c.d_perm;
  }
  hipError_t e = hipSuccess;
  auto conv = [&](int lo, int hi, int wi, const float* in, float* out, const float* res, float* xb, bool last) {
    if (e != hipSuccess) return;
    a.b_lo = lo;
    a.b_hi = hi;
    a.h_in = in;
    a.h_out = out;
    a.res = res;
    a.xb = xb;
    a.w = c.w_conv[wi];
    a.bias = c.w_bias[wi];
    a.logits = last ? logits : nullptr;
    ProfScope ps_(c, last ? RENO_K_CONV_LAST : RENO_K_CONV_MID);
    e = (C == 32) ? run_layer<32, false>(c, false, last, two, a) : run_layer<16, false>(c, false, last, two, a);
  };
  conv(n_lo, b_hi - 1, 0, c.h_c, c.h_b, nullptr, nullptr, false);
  conv(n_lo, b_hi - 1, 1, c.h_b, nullptr, c.h_c, c.h_d, false);
  conv(b_lo, b_hi, 2, c.h_d, c.h_b, nullptr, nullptr, false);
  conv(b_lo, b_hi, 3, c.h_b, c.h_a, c.h_d, nullptr, true);
  return e == hipSuccess ? hipGetLastError() : e;
}

// Full predictor with streamed weights (5x5x5 kernels or C above 32): the
// steps of launch_top on k_convw and a separate head launch.
template <int C, int KV>
hipError_t launch_top_wide(Ctx& c, int b_lo, int b_hi, float* logits, bool second) {
  const int b0 = c.b0();
  const int64_t ext_off = c.cap_model + 1;
  const RowMap rm{c.d_count, c.d_moff, (int64_t)c.cap_model, b0, ext_off, c.cap_rows()};
  const int n_lo = b_lo - 1;
  {
    ProfScope ps_(c, RENO_K_TOP_INPUT);
    const int blocks = (int)std::min<int64_t>(2048, (c.cap_rows() + 63) / 64);
    if (KV == 125)
      hipLaunchKernelGGL(k_top_prep5<C>, dim3(blocks), dim3(256), 0, c.stream, n_lo, b_hi - n_lo + 1, b_hi - n_lo,
                         b0, rm, c.lv_key, c.lv_code, (int64_t)c.cap_pts, c.d_hash, c.hash_lg, c.hreg(), c.fbits, c.w_embo,
                         c.d_nbr, c.h_c);
    else
      hipLaunchKernelGGL(k_top_prep<C>, dim3(blocks), dim3(256), 0, c.stream, n_lo, b_hi - n_lo + 1, b_hi - n_lo,
                         b0, rm, c.lv_key, c.lv_code, (int64_t)c.cap_pts, c.d_hash, c.hash_lg, c.hreg(), c.fbits, c.w_embo,
                         c.d_nbr, c.h_c);
  }
  ConvArgs a{};
  a.b0 = b0;
  a.count = c.d_count;
  a.moff = c.d_moff;
  a.cap_pts = c.cap_pts;
  a.cap_model = c.cap_model;
  a.lv_key = c.lv_key;
  a.nbr = c.d_nbr;
  a.hb = c.w_hbias;
  a.hw = c.w_head;
  a.lse = c.d_lse;
  a.err = c.d_err;
  a.emb = c.w_emb;
  a.s1_code = second ? c.lv_code : nullptr;
  a.lse2 = c.d_lse2;
  a.s1_out = c.d_s1;
  a.b_ext = b0;
  a.ext_off = ext_off;
  a.cap_rows = c.cap_rows();
  a.emb_d = c.w_embd;
  a.code = c.lv_code;
  a.fc = c.lv_fc;
  {  // tiles of voxels with similar neighbourhoods: smaller offset unions per tile and group
    ProfScope pso_(c, RENO_K_OTHER);
    const int nsc = b_hi - n_lo + 1;
    const int64_t windows = (c.cap_model + c.cap_pts + TO_W - 1) / TO_W + nsc;
    hipLaunchKernelGGL(k_tile_order, dim3((unsigned)windows), dim3(TO_THREADS), 0, c.stream, n_lo, nsc, rm,
                       KV == 125 ? 5 : 3, c.d_nbr, c.d_perm);
    a.perm = c.d_perm;
  }
  hipError_t e = hipSuccess;
  auto conv = [&](int lo, int hi, int wi, const float* in, float* out, const float* res, float* xb) {
    if (e != hipSuccess) return;
    a.b_lo = lo;
    a.b_hi = hi;
    a.h_in = in;
    a.h_out = out;
    a.res = res;
    a.xb = xb;
    a.w = c.w_conv[wi];
    a.bias = c.w_bias[wi];
    ProfScope ps_(c, RENO_K_CONV_MID);
    hipLaunchKernelGGL((k_convw<C, KV>), dim3(256), dim3(CW_THREADS), 0, c.stream, a);
    e = hipGetLastError();
  };
  conv(n_lo, b_hi - 1, 0, c.h_c, c.h_b, nullptr, nullptr);
  conv(n_lo, b_hi - 1, 1, c.h_b, nullptr, c.h_c, c.h_d);
  conv(b_lo, b_hi, 2, c.h_d, c.h_b, nullptr, nullptr);
  conv(b_lo, b_hi, 3, c.h_b, c.h_a, c.h_d, nullptr);
  if (e != hipSuccess) return e;
  {
    ProfScope ps_(c, RENO_K_CONV_LAST);
    a.b_lo = b_lo;
    a.b_hi = b_hi;
    a.h_in = c.h_a;
    a.logits = logits;
    if (c.p.head_mode == RENO_HEAD_TWO_STAGE) {
      constexpr int HT = headw_threads<C, true>();
      const int blocks = (int)std::min<int64_t>(4096, (c.cap_model + 16 * HT / 64 - 1) / (16 * HT / 64));
      hipLaunchKernelGGL((k_headw<C, true>), dim3(blocks), dim3(HT), 0, c.stream, a);
    } else {
      constexpr int HT = headw_threads<C, false>();
      const int blocks = (int)std::min<int64_t>(1024, (c.cap_model + 16 * HT / 64 - 1) / (16 * HT / 64));
      hipLaunchKernelGGL((k_headw<C, false>), dim3(blocks), dim3(HT), 0, c.stream, a);
    }
  }
  return hipGetLastError();
}

hipError_t launch_top_wide_any(Ctx& c, int b_lo, int b_hi, float* logits, bool second) {
  const bool k5 = c.ks() == 5;
  switch (c.p.channels) {
    case 16: return k5 ? launch_top_wide<16, 125>(c, b_lo, b_hi, logits, second)
                       : launch_top_wide<16, 27>(c, b_lo, b_hi, logits, second);
    case 32: return k5 ? launch_top_wide<32, 125>(c, b_lo, b_hi, logits, second)
                       : launch_top_wide<32, 27>(c, b_lo, b_hi, logits, second);
    case 64: return k5 ? launch_top_wide<64, 125>(c, b_lo, b_hi, logits, second)
                       : launch_top_wide<64, 27>(c, b_lo, b_hi, logits, second);
    default: return k5 ? launch_top_wide<128, 125>(c, b_lo, b_hi, logits, second)
                       : launch_top_wide<128, 27>(c, b_lo, b_hi, logits, second);
  }
}

hipError_t launch_model(Ctx& c, int b_lo, int b_hi, float* logits, bool second) {
  if (c.wide()) return launch_top_wide_any(c, b_lo, b_hi, logits, second);
  if (c.p.model_mode == RENO_MODEL_TOP) return launch_top(c, b_lo, b_hi, logits, second);
  ConvArgs a{};
  a.b_lo = b_lo;
  a.b_hi = b_hi;
  a.b0 = c.b0();
  a.count = c.d_count;
  a.moff = c.d_moff;
  a.cap_pts = c.cap_pts;
  a.cap_model = c.cap_model;
  a.lv_key = c.lv_key;
  a.lv_feat = c.lv_feat;
  a.hash = c.d_hash;
  a.hash_lg = c.hash_lg;
  a.hreg = c.hreg();
  a.fb = c.fbits;
  a.nbr = c.d_nbr;
  a.zero_feat = (int64_t)c.nlv * c.cap_pts;
  a.hb = c.w_hbias;
  a.hw = c.w_head;
  a.lse = c.d_lse;
  a.err = c.d_err;
  a.emb = c.w_emb;
  a.s1_code = second ? c.lv_code : nullptr;
  a.lse2 = c.d_lse2;
  a.s1_out = c.d_s1;
  const bool two = c.p.head_mode == RENO_HEAD_TWO_STAGE;
  const int L = c.p.layers;
  // sorted tiles where the launch is bound by matrix work: a batch of scales,
  // or the finest model scale (smaller scales are closer to latency-bound and
  // pay for the extra launch; on the 14-bit scan ordering the second finest
  // too cost 0.4 %, the third 1.5 %, none of the single scales 1.2 %)
  const bool order = L >= 2 && (b_lo != b_hi || b_lo >= c.B - 1);
  a.b_ext = -1;
  a.cap_rows = c.cap_model + 1;
  const RowMap rm{c.d_count, c.d_moff, (int64_t)c.cap_model, -1, 0, (int64_t)c.cap_model + 1};
  hipError_t e = hipSuccess;
  for (int l = 0; l < L && e == hipSuccess; ++l) {
    if (l == 1 && order) {
      ProfScope pso_(c, RENO_K_OTHER);
      const int nsc = b_hi - b_lo + 1;
      const int64_t windows = (c.cap_model + TO_W - 1) / TO_W + nsc;
      hipLaunchKernelGGL(k_tile_order, dim3((unsigned)windows), dim3(TO_THREADS), 0, c.stream, b_lo, nsc, rm, 3,
                         c.d_nbr, c.d_perm);
      a.perm = c.d_perm;
    }
    a.h_in = (l & 1) ? c.h_a : c.h_b;   // layer l reads what layer l-1 wrote
    a.h_out = (l & 1) ? c.h_b : c.h_a;  // layer 0 writes h_a
    a.w = c.w_conv[l];
    a.bias = c.w_bias[l];
    a.logits = (l == L - 1) ? logits : nullptr;
    const bool first = l == 0, last = l == L - 1;
    ProfScope ps_(c, last ? RENO_K_CONV_LAST : (first ? RENO_K_CONV_FIRST : RENO_K_CONV_MID), true);
    if (c.p.precision == RENO_PREC_BF16X3)
      e = (c.p.channels == 32) ? run_layer<32, true>(c, first, last, two, a)
                               : run_layer<16, true>(c, first, last, two, a);
    else
      e = (c.p.channels == 32) ? run_layer<32, false>(c, first, last, two, a)
                               : run_layer<16, false>(c, first, last, two, a);
  }
  return e;
}

hipError_t launch_head2(Ctx& c, int b, const uint8_t* s1, float* logits2) {
  ProfScope ps_(c, RENO_K_CONV_LAST);
  const bool bf = c.p.precision == RENO_PREC_BF16X3;
  const float* hw2 = c.w_head + (bf ? 64 * 8 : 64 * (c.p.channels / 4));
  const uint8_t* code = c.lv_code + c.lv(b);
  const int blocks = (int)std::min<int64_t>(1024, (c.cap_pts + 63) / 64);
#define RENO_HEAD2(CC, BFV)                                                                       \
  hipLaunchKernelGGL((k_head2<CC, BFV>), dim3(blocks), dim3(256), 0, c.stream, b, c.d_count, c.d_moff, \
                     (int64_t)c.cap_model, c.hlast(), s1, code, hw2, c.w_hbias + 16, c.w_emb, c.d_lse2, \
                     logits2, c.d_s1, c.d_err)
  if (c.p.channels == 128) {
    RENO_HEAD2(128, false);
  } else if (c.p.channels == 64) {
    RENO_HEAD2(64, false);
  } else if (c.p.channels == 32) {
    if (bf) RENO_HEAD2(32, true); else RENO_HEAD2(32, false);
  } else {
    if (bf) RENO_HEAD2(16, true); else RENO_HEAD2(16, false);
  }
#undef RENO_HEAD2
  return hipGetLastError();
}

}  // namespace reno
