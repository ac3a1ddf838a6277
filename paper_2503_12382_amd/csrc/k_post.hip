// Code lengths (Eq. 4), the quantised distributions handed to the host
// arithmetic coder, and the getters that copy per-scale arrays out of the
// context.  All sizes are read from the device.

#include "ctx.h"

namespace reno {
namespace {

constexpr float INV_LN2 = 1.4426950408889634f;

// bits_v = (lse_v - z_{O_b[v]}) / ln 2 with z_o = hb[o] + sum_c H[c][o] h_L[v][c]
// (fp32, channel order).  Two-stage head (TWO): with a = O & 15, s = O >> 4,
// bits_v = ((lse1_v - z1_a) + (lse2_v - z2_s)) / ln 2, z1_a = hb1[a] +
// sum_c H1[c][a] h[c], z2_s = hb2[s] + sum_c H2[c][s] (h[c] + E[a][c]).
// Blocks stage the transposed head HT [NS][C] in LDS once (rows padded by one
// word so that lanes reading different symbols hit different banks), then
// waves take chunks of 64 voxels (one per lane) over all scales of the
// launch.  Each chunk's sum in double goes to partial[b][chunk], and a second
// one-wave-per-scale kernel sums them in chunk order (lane-strided, then a
// fixed xor tree): deterministic.  The kernel boundary publishes the partials;
// a device-scope fence inside the kernel would write back the whole L2 of the
// XCD and costs more than the second launch.
constexpr int CL_THREADS = 1024;
constexpr int CL_CHUNK = 64;

template <int C, bool TWO>
__global__ void __launch_bounds__(CL_THREADS) k_code_length(
    int b_lo, int nsc, int b0, const int32_t* __restrict__ count, const int32_t* __restrict__ moff,
    int64_t cap_pts, int64_t cap_model, const uint8_t* __restrict__ lv_code,
    const float* __restrict__ hL, const float* __restrict__ HT, const float* __restrict__ hb,
    const float* __restrict__ lse, const float* __restrict__ lse2, const float* __restrict__ emb,
    float* __restrict__ bits_out, double* partial, int max_chunks) {
  constexpr int NS = TWO ? 32 : 256;
  constexpr int RS = C + 1;  // padded LDS row
  __shared__ float s_HT[NS * RS];
  __shared__ float s_hb[NS];
  __shared__ float s_emb[TWO ? 16 * C : 1];
  __shared__ int64_t s_cpre[NLEV + 1];  // chunk prefix over the launch's scales
  __shared__ int64_t s_n[NLEV], s_mo[NLEV];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  static_assert(NLEV < 32, "the scale scan covers 32 lanes");
  if (w == 0) {  // sizes of all scales loaded at once (lane i: scale b_lo + i), prefix by a lane scan
    int64_t n = 0, mo = 0;
    if (lane < nsc) {
      n = count[b_lo + lane];
      mo = moff[b_lo + lane];
      if (mo + n > cap_model) n = 0;  // capacity overflow, latched where the size was made
    }
    const int nc = (int)((n + CL_CHUNK - 1) / CL_CHUNK);
    int incl = nc;
#pragma unroll
    for (int o = 1; o < 32; o <<= 1) {
      const int y = __shfl_up(incl, o);
      if (lane >= o) incl += y;
    }
    if (lane <= nsc) s_cpre[lane] = incl - nc;
    if (lane < nsc) {
      s_n[lane] = n;
      s_mo[lane] = mo;
    }
  }
  {  // staging: every load of a thread issued before its stores
    constexpr int PER = (NS * C + CL_THREADS - 1) / CL_THREADS;
    float t[PER];
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = k * CL_THREADS + tid;
      t[k] = i < NS * C ? HT[i] : 0.0f;
    }
#pragma unroll
    for (int k = 0; k < PER; ++k) {
      const int i = k * CL_THREADS + tid;
      if (i < NS * C) s_HT[(i / C) * RS + (i % C)] = t[k];
    }
  }
  for (int i = tid; i < NS; i += CL_THREADS) s_hb[i] = hb[i];
  if constexpr (TWO)
    for (int i = tid; i < 16 * C; i += CL_THREADS) s_emb[i] = emb[i];
  __syncthreads();
  const int64_t nchunks_all = s_cpre[nsc];
  const int64_t waves = (int64_t)gridDim.x * (CL_THREADS / 64);
  for (int64_t ch = (int64_t)blockIdx.x * (CL_THREADS / 64) + w; ch < nchunks_all; ch += waves) {
    int si = 0;
    while (si + 1 < nsc && s_cpre[si + 1] <= ch) ++si;
    const int b = b_lo + si;
    const int64_t mo = s_mo[si];
    const int64_t n = s_n[si];
    const int64_t cib = ch - s_cpre[si];  // chunk index inside the scale
    const int64_t v = cib * CL_CHUNK + lane;
    const int64_t vv = v < n ? v : n - 1;  // clamped: every load is issued
    const int o = lv_code[(int64_t)(b - b0) * cap_pts + vv];
    const float l1 = lse[mo + vv];
    const float l2 = TWO ? lse2[mo + vv] : 0.0f;
    // the row in chunks of HC channels (all of it for C <= 32); the dot
    // products run over c in ascending order either way
    constexpr int HC = C <= 32 ? C : 16;
    const float4* hr = reinterpret_cast<const float4*>(hL + (mo + vv) * C);
    float bt;
    const int a1 = o & 15, a2 = 16 + (o >> 4);
    float z1 = TWO ? s_hb[a1] : s_hb[o], z2 = TWO ? s_hb[a2] : 0.0f;
#pragma unroll
    for (int c0 = 0; c0 < C; c0 += HC) {
      float h[HC];
#pragma unroll
      for (int c4 = 0; c4 < HC / 4; ++c4) {
        const float4 t = hr[c0 / 4 + c4];
        h[4 * c4] = t.x;
        h[4 * c4 + 1] = t.y;
        h[4 * c4 + 2] = t.z;
        h[4 * c4 + 3] = t.w;
      }
#pragma unroll
      for (int cc = 0; cc < HC; ++cc) {
        const int c = c0 + cc;
        if constexpr (TWO) {
          z1 = fmaf(s_HT[a1 * RS + c], h[cc], z1);
          z2 = fmaf(s_HT[a2 * RS + c], h[cc] + s_emb[a1 * C + c], z2);
        } else {
          z1 = fmaf(s_HT[o * RS + c], h[cc], z1);
        }
      }
    }
    if constexpr (TWO)
      bt = ((l1 - z1) + (l2 - z2)) * INV_LN2;
    else
      bt = (l1 - z1) * INV_LN2;
    double acc = 0.0;
    if (v < n) {
      if (bits_out) bits_out[mo - s_mo[0] + v] = bt;
      acc = (double)bt;
    }
    for (int d = 32; d > 0; d >>= 1) acc += __shfl_xor(acc, d);
    if (lane == 0) partial[(int64_t)b * max_chunks + cib] = acc;
  }
}

// Per-scale totals from the chunk partials: one block of 256 threads per
// scale; thread t adds chunks t, t+256, ... in order (loads issued in batches
// before the adds), then a fixed tree: xor within each wave, waves in order.
__global__ void __launch_bounds__(256) k_bits_total(int b_lo, const int32_t* __restrict__ count,
                                                    const int32_t* __restrict__ moff, int64_t cap_model,
                                                    const double* __restrict__ partial, int max_chunks,
                                                    double* __restrict__ total) {
  __shared__ double s_w[4];
  const int b = b_lo + blockIdx.x, tid = threadIdx.x;
  int64_t n = count[b];
  if (moff[b] + n > cap_model) n = 0;
  const int64_t nch = (n + CL_CHUNK - 1) / CL_CHUNK;
  const double* p = partial + (int64_t)b * max_chunks;
  double t = 0.0;
  constexpr int BATCH = 8;
  for (int64_t i0 = tid; i0 < nch; i0 += 256 * BATCH) {
    double x[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int64_t i = i0 + (int64_t)k * 256;
      x[k] = i < nch ? p[i] : 0.0;
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) t += x[k];
  }
  for (int d = 32; d > 0; d >>= 1) t += __shfl_xor(t, d);
  if ((tid & 63) == 0) s_w[tid >> 6] = t;
  __syncthreads();
  if (tid == 0) total[b] = (s_w[0] + s_w[1]) + (s_w[2] + s_w[3]);
}

// Quantised distributions for the host coder (Sec. 3, Eq. 4 made concrete):
// over K symbols, f_s = 1 + floor(p_s * (2^16 - 2K)) in fp32 with p_s =
// exp(z_s - lse) and z_s recomputed from h_L in channel order; the leftover
// 2^16 - sum f goes to the lowest-index largest f_s, so sum f = 2^16 and every
// f_s >= 1.  Encoder intervals and decoder tables come from the same code and
// inputs, so they agree bit for bit.

// 256-symbol table of one voxel in one wavefront: lane l ends with the final
// frequencies of symbols 4l .. 4l+3.
__device__ __forceinline__ void table256(const float* __restrict__ h, float l, const float* __restrict__ H,
                                         const float* __restrict__ hb, int C, int lane, uint32_t (&f)[4]) {
  uint32_t sum = 0, best = 0;
  int besti = 0;
  for (int e = 0; e < 4; ++e) {
    const int s = lane * 4 + e;
    float z = hb[s];
    for (int c = 0; c < C; ++c) z = fmaf(H[c * 256 + s], h[c], z);
    const float p = __expf(z - l);
    f[e] = 1u + (uint32_t)floorf(p * 65024.0f);
    sum += f[e];
    if (f[e] > best) {
      best = f[e];
      besti = s;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    sum += (uint32_t)__shfl_xor((int)sum, o);
    const uint32_t ob = (uint32_t)__shfl_xor((int)best, o);
    const int oi = __shfl_xor(besti, o);
    if (ob > best || (ob == best && oi < besti)) {
      best = ob;
      besti = oi;
    }
  }
  const uint32_t left = 65536u - sum;
  for (int e = 0; e < 4; ++e) f[e] += (lane * 4 + e == besti) ? left : 0u;
}

// 16-symbol table of one voxel over 16 consecutive lanes (s = lane % 16): the
// stage-1 or stage-2 distribution of the two-stage head.  Hp is the plain
// [C][32] table of both stages (column col0 + s), emb_row the Emb(S1) row added
// to h for stage 2 (NULL for stage 1).  Returns f_s.
__device__ __forceinline__ uint32_t table16(const float* __restrict__ h, const float* __restrict__ emb_row,
                                            float l, const float* __restrict__ Hp, int col0,
                                            const float* __restrict__ hb, int C, int s) {
  float z = hb[col0 + s];
  for (int c = 0; c < C; ++c) z = fmaf(Hp[c * 32 + col0 + s], emb_row ? h[c] + emb_row[c] : h[c], z);
  const float p = __expf(z - l);
  uint32_t f = 1u + (uint32_t)floorf(p * 65504.0f);
  uint32_t sum = f, best = f;
  int besti = s;
  for (int o = 1; o < 16; o <<= 1) {
    sum += (uint32_t)__shfl_xor((int)sum, o);
    const uint32_t ob = (uint32_t)__shfl_xor((int)best, o);
    const int oi = __shfl_xor(besti, o);
    if (ob > best || (ob == best && oi < besti)) {
      best = ob;
      besti = oi;
    }
  }
  return f + (s == besti ? 65536u - sum : 0u);
}

// exclusive prefix of v over the 16-lane group of this lane
__device__ __forceinline__ uint32_t excl16(uint32_t v, int s) {
  uint32_t inc = v;
  for (int o = 1; o < 16; o <<= 1) {
    const uint32_t t = (uint32_t)__shfl_up((int)inc, o, 16);
    if (s >= o) inc += t;
  }
  return inc - v;
}

// One-stage tables [N][256] of one scale: one wavefront per voxel.
__global__ void __launch_bounds__(256) k_symbol_freqs(const int32_t* __restrict__ count,
                                                      const int32_t* __restrict__ moff, int b,
                                                      int64_t cap_model,
                                                      const float* __restrict__ hL, int C,
                                                      const float* __restrict__ H,
                                                      const float* __restrict__ hb,
                                                      const float* __restrict__ lse,
                                                      uint16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t wstride = (int64_t)gridDim.x * (blockDim.x / 64);
  for (int64_t v = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6); v < n; v += wstride) {
    uint32_t f[4];
    table256(hL + (mo + v) * C, lse[mo + v], H, hb, C, lane, f);
    uint16_t* dst = out + v * 256 + lane * 4;
    for (int e = 0; e < 4; ++e) dst[e] = (uint16_t)f[e];
  }
}

// One-stage cumulative tables [N][256]: the start of every symbol in the
// voxel's table (exclusive prefix of the frequencies), one wavefront per voxel.
__global__ void __launch_bounds__(256) k_symbol_cdf(const int32_t* __restrict__ count,
                                                    const int32_t* __restrict__ moff, int b,
                                                    int64_t cap_model,
                                                    const float* __restrict__ hL, int C,
                                                    const float* __restrict__ H,
                                                    const float* __restrict__ hb,
                                                    const float* __restrict__ lse,
                                                    uint16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t wstride = (int64_t)gridDim.x * (blockDim.x / 64);
  for (int64_t v = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6); v < n; v += wstride) {
    uint32_t f[4];
    table256(hL + (mo + v) * C, lse[mo + v], H, hb, C, lane, f);
    const uint32_t mine = f[0] + f[1] + f[2] + f[3];
    uint32_t inc = mine;
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t t = (uint32_t)__shfl_up((int)inc, d);
      if (lane >= d) inc += t;
    }
    uint32_t st = inc - mine;
    uint16_t* dst = out + v * 256 + lane * 4;
    for (int e = 0; e < 4; ++e) {
      dst[e] = (uint16_t)st;
      st += f[e];
    }
  }
}

// Two-stage cumulative tables [N][16] of one scale and stage: 4 voxels per
// wavefront, the same tables as k_symbol_freqs16 summed over the 16 lanes.
__global__ void __launch_bounds__(256) k_symbol_cdf16(const int32_t* __restrict__ count,
                                                      const int32_t* __restrict__ moff, int b, int stage,
                                                      int64_t cap_model, const float* __restrict__ hL, int C,
                                                      const float* __restrict__ Hp, const float* __restrict__ hb,
                                                      const float* __restrict__ emb, const uint8_t* __restrict__ s1,
                                                      const float* __restrict__ lse, const float* __restrict__ lse2,
                                                      uint16_t* __restrict__ out) {
  const int s = threadIdx.x & 15;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t gstride = (int64_t)gridDim.x * (blockDim.x / 16);
  for (int64_t v0 = (int64_t)blockIdx.x * (blockDim.x / 16); v0 < n; v0 += gstride) {
    // the whole wavefront runs the shuffles; lanes past the last voxel write nothing
    const int64_t v = v0 + (threadIdx.x >> 4);
    const int64_t pr = mo + (v < n ? v : n - 1);
    const float* h = hL + pr * C;
    const uint32_t f = stage == 1 ? table16(h, nullptr, lse[pr], Hp, 0, hb, C, s)
                                  : table16(h, emb + (int)s1[pr] * C, lse2[pr], Hp, 16, hb, C, s);
    const uint32_t st = excl16(f, s);
    if (v < n) out[v * 16 + s] = (uint16_t)st;
  }
}

// One-stage encoder intervals [N][2] = (start, freq) of O_b[v] in its table.
__global__ void __launch_bounds__(256) k_symbol_intervals(const int32_t* __restrict__ count,
                                                          const int32_t* __restrict__ moff, int b, int b_lo,
                                                          int64_t cap_model, const uint8_t* __restrict__ code,
                                                          const float* __restrict__ hL, int C,
                                                          const float* __restrict__ H,
                                                          const float* __restrict__ hb,
                                                          const float* __restrict__ lse,
                                                          uint16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t wstride = (int64_t)gridDim.x * (blockDim.x / 64);
  for (int64_t v = (int64_t)blockIdx.x * (blockDim.x / 64) + (threadIdx.x >> 6); v < n; v += wstride) {
    uint32_t f[4];
    table256(hL + (mo + v) * C, lse[mo + v], H, hb, C, lane, f);
    const int o = code[v];
    const uint32_t mine = f[0] + f[1] + f[2] + f[3];
    uint32_t inc = mine;  // inclusive prefix over lanes
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t t = (uint32_t)__shfl_up((int)inc, d);
      if (lane >= d) inc += t;
    }
    if (lane == (o >> 2)) {
      uint32_t st = inc - mine;
      for (int e = 0; e < (o & 3); ++e) st += f[e];
      const int64_t ro = mo - moff[b_lo] + v;  // row in the concatenated output
      out[ro * 2] = (uint16_t)st;
      out[ro * 2 + 1] = (uint16_t)f[o & 3];
    }
  }
}

// Two-stage tables [N][16] of one scale and stage: 4 voxels per wavefront.
__global__ void __launch_bounds__(256) k_symbol_freqs16(const int32_t* __restrict__ count,
                                                        const int32_t* __restrict__ moff, int b, int stage,
                                                        int64_t cap_model, const float* __restrict__ hL, int C,
                                                        const float* __restrict__ Hp, const float* __restrict__ hb,
                                                        const float* __restrict__ emb, const uint8_t* __restrict__ s1,
                                                        const float* __restrict__ lse, const float* __restrict__ lse2,
                                                        uint16_t* __restrict__ out) {
  const int s = threadIdx.x & 15;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t gstride = (int64_t)gridDim.x * (blockDim.x / 16);
  for (int64_t v = (int64_t)blockIdx.x * (blockDim.x / 16) + (threadIdx.x >> 4); v < n; v += gstride) {
    const int64_t pr = mo + v;
    const float* h = hL + pr * C;
    const uint32_t f = stage == 1 ? table16(h, nullptr, lse[pr], Hp, 0, hb, C, s)
                                  : table16(h, emb + (int)s1[pr] * C, lse2[pr], Hp, 16, hb, C, s);
    out[v * 16 + s] = (uint16_t)f;
  }
}

// Two-stage encoder intervals [N][4]: (start, freq) of S1 = O & 15 in the
// stage-1 table, then of S2 = O >> 4 in the stage-2 table given that S1.
__global__ void __launch_bounds__(256) k_symbol_intervals16(const int32_t* __restrict__ count,
                                                            const int32_t* __restrict__ moff, int b, int b_lo,
                                                            int64_t cap_model, const uint8_t* __restrict__ code,
                                                            const float* __restrict__ hL, int C,
                                                            const float* __restrict__ Hp,
                                                            const float* __restrict__ hb,
                                                            const float* __restrict__ emb,
                                                            const float* __restrict__ lse,
                                                            const float* __restrict__ lse2,
                                                            uint16_t* __restrict__ out) {
  const int s = threadIdx.x & 15;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t gstride = (int64_t)gridDim.x * (blockDim.x / 16);
  for (int64_t v = (int64_t)blockIdx.x * (blockDim.x / 16) + (threadIdx.x >> 4); v < n; v += gstride) {
    const int64_t pr = mo + v;
    const float* h = hL + pr * C;
    const int o = code[v], a1 = o & 15, a2 = o >> 4;
    const uint32_t f1 = table16(h, nullptr, lse[pr], Hp, 0, hb, C, s);
    const uint32_t st1 = excl16(f1, s);
    const uint32_t f2 = table16(h, emb + a1 * C, lse2[pr], Hp, 16, hb, C, s);
    const uint32_t st2 = excl16(f2, s);
    const int64_t ro = mo - moff[b_lo] + v;  // row in the concatenated output
    if (s == a1) {
      out[ro * 4] = (uint16_t)st1;
      out[ro * 4 + 1] = (uint16_t)f1;
    }
    if (s == a2) {
      out[ro * 4 + 2] = (uint16_t)st2;
      out[ro * 4 + 3] = (uint16_t)f2;
    }
  }
}

// ---- the same tables with the head held in registers (C = 16 or 32) ----
// One wavefront per voxel for 256 symbols, four voxels per wavefront (16
// lanes each) for 16; each lane keeps its symbols' head columns in registers
// for the whole launch and the voxel's row h_L is read once per wavefront
// (uniform loads).  Logits accumulate over c in ascending order exactly as in
// table256 / table16, so every table is bit-identical to theirs.
// TB_ENTRY: the decoder's entries, uint32 start | f << 16 per symbol
enum { TB_FREQ = 0, TB_CDF = 1, TB_IV = 2, TB_ENTRY = 3 };

__device__ __forceinline__ int uniform_wave() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// DPP lane moves (CDNA): row_shr:k (0x110 + k) takes the value of lane
// l - k of the same 16-lane row, row_ror:k (0x120 + k) of lane l - k mod 16
// of the row, row_bcast:15 (0x142) lane 15 of the previous row, row_bcast:31
// (0x143) lane 31.  Lanes whose source lies outside are fixed by the callers.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, CTRL, 0xF, 0xF, false);
}

// The moves run in every lane and their results are masked with bit
// operations: a move under a lane mask would read disabled source lanes.
__device__ __forceinline__ uint32_t keep(bool c) { return c ? 0xFFFFFFFFu : 0u; }

// inclusive prefix sum over the 64 lanes
__device__ __forceinline__ uint32_t scan_add64(uint32_t v, int lane) {
  const int r = lane & 15;
  v += dpp<0x111>(v) & keep(r >= 1);
  v += dpp<0x112>(v) & keep(r >= 2);
  v += dpp<0x114>(v) & keep(r >= 4);
  v += dpp<0x118>(v) & keep(r >= 8);
  v += dpp<0x142>(v) & keep((lane & 31) >= 16);
  v += dpp<0x143>(v) & keep(lane >= 32);
  return v;
}

// running maximum over the 64 lanes (lane 63 ends with the maximum)
__device__ __forceinline__ uint32_t scan_max64(uint32_t v, int lane) {
  const int r = lane & 15;
  v = max(v, dpp<0x111>(v) & keep(r >= 1));
  v = max(v, dpp<0x112>(v) & keep(r >= 2));
  v = max(v, dpp<0x114>(v) & keep(r >= 4));
  v = max(v, dpp<0x118>(v) & keep(r >= 8));
  v = max(v, dpp<0x142>(v) & keep((lane & 31) >= 16));
  v = max(v, dpp<0x143>(v) & keep(lane >= 32));
  return v;
}

// Quantisation of table256 from the logits of symbols 4 lane .. 4 lane + 3:
// f_s = 1 + floor(p_s (2^16 - 512)), the leftover 2^16 - sum f to the
// lowest-index largest f_s.  Returns the final f of the lane's symbols and
// the start (sum of the final f below) of its first symbol.
__device__ __forceinline__ uint32_t quantise256(const float (&z)[4], float l, int lane, uint32_t (&f)[4]) {
  uint32_t lmax = 0, lsum = 0;
  int lidx = 0;
  for (int e = 0; e < 4; ++e) {
    const float p = __expf(z[e] - l);
    f[e] = 1u + (uint32_t)floorf(p * 65024.0f);
    lsum += f[e];
    if (f[e] > lmax) {
      lmax = f[e];
      lidx = e;
    }
  }
  const uint32_t incl = scan_add64(lsum, lane);
  const uint32_t total = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
  const uint32_t gmax = (uint32_t)__builtin_amdgcn_readlane((int)scan_max64(lmax, lane), 63);
  const uint64_t ball = __ballot(lmax == gmax);
  const int l0 = __ffsll((long long)ball) - 1;  // lowest lane holding the maximum
  const int besti = 4 * l0 + __builtin_amdgcn_readlane(lidx, l0);
  const uint32_t left = 65536u - total;
  for (int e = 0; e < 4; ++e) f[e] += (4 * lane + e == besti) ? left : 0u;
  return incl - lsum + (besti < 4 * lane ? left : 0u);
}

template <int C, int MODE>
__global__ void __launch_bounds__(256) k_table256r(const int32_t* __restrict__ count,
                                                   const int32_t* __restrict__ moff, int b, int b_lo,
                                                   int64_t cap_model, const uint8_t* __restrict__ code,
                                                   const float* __restrict__ hL, const float* __restrict__ H,
                                                   const float* __restrict__ hb, const float* __restrict__ lse,
                                                   uint16_t* __restrict__ out) {
  const int lane = threadIdx.x & 63;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t wstride = (int64_t)gridDim.x * (blockDim.x / 64);
  const int64_t v_first = (int64_t)blockIdx.x * (blockDim.x / 64) + uniform_wave();
  if (v_first >= n) return;  // no voxel for this wavefront: the head is not loaded
  float w[C][4];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    const float4 t = reinterpret_cast<const float4*>(H + c * 256)[lane];
    w[c][0] = t.x;
    w[c][1] = t.y;
    w[c][2] = t.z;
    w[c][3] = t.w;
  }
  const float4 bias = reinterpret_cast<const float4*>(hb)[lane];
  for (int64_t v = v_first; v < n; v += wstride) {
    const float* h = hL + (mo + v) * C;
    float z[4] = {bias.x, bias.y, bias.z, bias.w};
#pragma unroll
    for (int c = 0; c < C; ++c) {
      const float hc = h[c];
#pragma unroll
      for (int e = 0; e < 4; ++e) z[e] = fmaf(w[c][e], hc, z[e]);
    }
    uint32_t f[4];
    uint32_t st = quantise256(z, lse[mo + v], lane, f);
    if constexpr (MODE == TB_FREQ) {
      uint16_t* dst = out + v * 256 + lane * 4;
      for (int e = 0; e < 4; ++e) dst[e] = (uint16_t)f[e];
    } else {
      if constexpr (MODE == TB_CDF) {
        uint16_t* dst = out + v * 256 + lane * 4;
        for (int e = 0; e < 4; ++e) {
          dst[e] = (uint16_t)st;
          st += f[e];
        }
      } else if constexpr (MODE == TB_ENTRY) {
        uint4 ent;
        ent.x = st | (f[0] << 16);
        st += f[0];
        ent.y = st | (f[1] << 16);
        st += f[1];
        ent.z = st | (f[2] << 16);
        st += f[2];
        ent.w = st | (f[3] << 16);
        reinterpret_cast<uint4*>(out)[v * 64 + lane] = ent;
      } else {
        const int o = code[v];
        if (lane == (o >> 2)) {
          for (int e = 0; e < (o & 3); ++e) st += f[e];
          const int64_t ro = mo - moff[b_lo] + v;  // row in the concatenated output
          out[ro * 2] = (uint16_t)st;
          out[ro * 2 + 1] = (uint16_t)f[o & 3];
        }
      }
    }
  }
}

// 16-symbol table of the voxel of this lane's row (16 lanes, s = lane % 16)
// from its logit z (the quantisation of table16): returns f_s and its
// exclusive start in the row.  Row totals by rotations, the start by row
// shifts.
__device__ __forceinline__ uint32_t quantise16(float z, float l, int lane, uint32_t* start) {
  const int s = lane & 15;
  const float p = __expf(z - l);
  uint32_t f = 1u + (uint32_t)floorf(p * 65504.0f);
  uint32_t sum = f, mx = f;
  sum += dpp<0x128>(sum);  // row_ror:8, 4, 2, 1: every lane ends with the row total
  sum += dpp<0x124>(sum);
  sum += dpp<0x122>(sum);
  sum += dpp<0x121>(sum);
  mx = max(mx, dpp<0x128>(mx));
  mx = max(mx, dpp<0x124>(mx));
  mx = max(mx, dpp<0x122>(mx));
  mx = max(mx, dpp<0x121>(mx));
  // the lowest symbol of the row holding the maximum
  const uint64_t ball = __ballot(f == mx);
  const uint32_t rowbits = (uint32_t)(ball >> (lane & 48)) & 0xFFFFu;
  const int besti = __ffs(rowbits) - 1;
  const uint32_t left = 65536u - sum;
  f += s == besti ? left : 0u;
  uint32_t inc = f;  // inclusive prefix within the row
  inc += dpp<0x111>(inc) & keep(s >= 1);
  inc += dpp<0x112>(inc) & keep(s >= 2);
  inc += dpp<0x114>(inc) & keep(s >= 4);
  inc += dpp<0x118>(inc) & keep(s >= 8);
  *start = inc - f;
  return f;
}

// Two-stage tables: STAGE 1 or 2 (MODE TB_FREQ / TB_CDF), or both stages'
// encoder intervals (MODE TB_IV, STAGE ignored).
template <int C, int MODE, int STAGE>
__global__ void __launch_bounds__(256) k_table16r(const int32_t* __restrict__ count,
                                                  const int32_t* __restrict__ moff, int b, int b_lo,
                                                  int64_t cap_model, const uint8_t* __restrict__ code,
                                                  const float* __restrict__ hL, const float* __restrict__ Hp,
                                                  const float* __restrict__ hb, const float* __restrict__ emb,
                                                  const uint8_t* __restrict__ s1, const float* __restrict__ lse,
                                                  const float* __restrict__ lse2, uint16_t* __restrict__ out) {
  constexpr bool ONE = MODE == TB_IV || STAGE == 1;
  constexpr bool TWO = MODE == TB_IV || STAGE == 2;
  const int s = threadIdx.x & 15;
  const int64_t mo = moff[b];
  int64_t n = count[b];
  if (mo + n > cap_model) n = 0;
  const int64_t gstride = (int64_t)gridDim.x * (blockDim.x / 16);
  const int64_t v_first = (int64_t)blockIdx.x * (blockDim.x / 16) + 4 * uniform_wave();
  if (v_first >= n) return;  // no voxel for this wavefront: the head is not loaded
  float w1[ONE ? C : 1], w2[TWO ? C : 1];
#pragma unroll
  for (int c = 0; c < C; ++c) {
    if constexpr (ONE) w1[c] = Hp[c * 32 + s];
    if constexpr (TWO) w2[c] = Hp[c * 32 + 16 + s];
  }
  const float b1 = ONE ? hb[s] : 0.0f, b2 = TWO ? hb[16 + s] : 0.0f;
  for (int64_t v0 = v_first; v0 < n; v0 += gstride) {
    // the whole wavefront runs the shuffles; groups past the last voxel write nothing
    const int64_t v = v0 + ((threadIdx.x >> 4) & 3);
    const int64_t pr = mo + (v < n ? v : n - 1);
    const float* h = hL + pr * C;
    const int o = MODE == TB_IV ? (int)code[v < n ? v : n - 1] : 0;
    const int lane = threadIdx.x & 63;
    uint32_t f1 = 0, f2 = 0, st1 = 0, st2 = 0;
    if constexpr (ONE) {
      float z = b1;
#pragma unroll
      for (int c = 0; c < C; ++c) z = fmaf(w1[c], h[c], z);
      f1 = quantise16(z, lse[pr], lane, &st1);
    }
    if constexpr (TWO) {
      const int a1 = MODE == TB_IV ? (o & 15) : (int)s1[pr];
      const float* e = emb + a1 * C;
      float z = b2;
#pragma unroll
      for (int c = 0; c < C; ++c) z = fmaf(w2[c], h[c] + e[c], z);
      f2 = quantise16(z, lse2[pr], lane, &st2);
    }
    if constexpr (MODE == TB_FREQ) {
      if (v < n) out[v * 16 + s] = (uint16_t)(STAGE == 1 ? f1 : f2);
    } else if constexpr (MODE == TB_CDF) {
      if (v < n) out[v * 16 + s] = (uint16_t)(STAGE == 1 ? st1 : st2);
    } else if constexpr (MODE == TB_ENTRY) {
      const uint32_t f = STAGE == 1 ? f1 : f2, st = STAGE == 1 ? st1 : st2;
      if (v < n) reinterpret_cast<uint32_t*>(out)[v * 16 + s] = st | (f << 16);
    } else {
      const int64_t ro = mo - moff[b_lo] + v;  // row in the concatenated output
      if (v < n && s == (o & 15)) {
        out[ro * 4] = (uint16_t)st1;
        out[ro * 4 + 1] = (uint16_t)f1;
      }
      if (v < n && s == (o >> 4)) {
        out[ro * 4 + 2] = (uint16_t)st2;
        out[ro * 4 + 3] = (uint16_t)f2;
      }
    }
  }
}

// Cumulative tables [N][K] to the decoder's entries start | f << 16.
__global__ void k_cdf_entries(const int32_t* __restrict__ count, int b, int K, const uint16_t* __restrict__ start,
                              uint32_t* __restrict__ entries) {
  const int64_t n = (int64_t)count[b] * K;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x) {
    const uint32_t st = start[i];
    const uint32_t nx = (i % K) + 1 < K ? (uint32_t)start[i + 1] : 65536u;
    entries[i] = st | ((nx - st) << 16);
  }
}

__global__ void k_coords(const uint64_t* __restrict__ key, const int32_t* __restrict__ count, int b,
                         int32_t* __restrict__ xyz, uint64_t* __restrict__ keys) {
  const int64_t n = count[b];
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const uint64_t kf = key[i];
    if (keys) keys[i] = kf;  // with the frame id of a batch above the Morton bits
    const uint64_t k = morton_part(kf, b);
    if (xyz) {
      xyz[3 * i + 0] = (int32_t)compact3(k);
      xyz[3 * i + 1] = (int32_t)compact3(k >> 1);
      xyz[3 * i + 2] = (int32_t)compact3(k >> 2);
    }
  }
}

__global__ void k_copy_u8(const uint8_t* __restrict__ src, const int32_t* __restrict__ count, int b,
                          uint8_t* __restrict__ dst) {
  const int64_t n = count[b];
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

__global__ void k_copy_i32(const int32_t* __restrict__ src, const int32_t* __restrict__ count,
                           int b, int mult, int32_t* __restrict__ dst) {
  const int64_t n = (int64_t)count[b] * mult;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = src[i];
}

// neighbour map rows of scale b start at its packed model row (device value)
__global__ void k_copy_map(const int32_t* __restrict__ nbr, const int32_t* __restrict__ moff,
                           const int32_t* __restrict__ count, int b, int64_t cap_model, int kv, int stride,
                           int32_t* __restrict__ dst) {
  int64_t n = (int64_t)count[b];
  if (moff[b] + n > cap_model) n = 0;
  n *= kv;
  const int64_t o = (int64_t)moff[b] * stride;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    dst[i] = nbr[o + (i / kv) * stride + i % kv];
}

unsigned grid_for(int64_t cap, int per_block) {
  int64_t g = (cap + per_block - 1) / per_block;
  if (g > 2048) g = 2048;
  if (g < 1) g = 1;
  return (unsigned)g;
}

}  // namespace

template <int C, bool TWO>
void run_code_length(Ctx& c, int b_lo, int b_hi, float* bits) {
  const int max_chunks = (int)((c.cap_pts + CL_CHUNK - 1) / CL_CHUNK);
  // one block per CU at most; small batches need fewer
  const int64_t chunks = (int64_t)(b_hi - b_lo + 1) * max_chunks;
  const int blocks = (int)std::min<int64_t>(256, (chunks + CL_THREADS / 64 - 1) / (CL_THREADS / 64));
  hipLaunchKernelGGL((k_code_length<C, TWO>), dim3(blocks), dim3(CL_THREADS), 0, c.stream, b_lo,
                     b_hi - b_lo + 1, c.b0(), c.d_count, c.d_moff, c.cap_pts, c.cap_model, c.lv_code,
                     c.hlast(), c.w_head_t, c.w_hbias, c.d_lse, c.d_lse2, c.w_emb, bits, c.d_partial,
                     max_chunks);
  hipLaunchKernelGGL(k_bits_total, dim3(b_hi - b_lo + 1), dim3(256), 0, c.stream, b_lo, c.d_count, c.d_moff,
                     (int64_t)c.cap_model, c.d_partial, max_chunks, c.d_total);
}

hipError_t launch_code_length(Ctx& c, int b_lo, int b_hi, float* bits) {
  ProfScope ps_(c, RENO_K_CODE_LENGTH);
  const bool two = c.p.head_mode == RENO_HEAD_TWO_STAGE;
  switch (c.p.channels) {
    case 128:
      two ? run_code_length<128, true>(c, b_lo, b_hi, bits) : run_code_length<128, false>(c, b_lo, b_hi, bits);
      break;
    case 64:
      two ? run_code_length<64, true>(c, b_lo, b_hi, bits) : run_code_length<64, false>(c, b_lo, b_hi, bits);
      break;
    case 32:
      two ? run_code_length<32, true>(c, b_lo, b_hi, bits) : run_code_length<32, false>(c, b_lo, b_hi, bits);
      break;
    default:
      two ? run_code_length<16, true>(c, b_lo, b_hi, bits) : run_code_length<16, false>(c, b_lo, b_hi, bits);
  }
  return hipGetLastError();
}

// register-resident table kernels: C = 16 or 32; wavefronts of 64 voxels
// (256 symbols) or 256 voxels (16 symbols) each, up to 2048 workgroups
template <int C>
void run_table256r(Ctx& c, int mode, int b, int b_lo, const uint8_t* code, uint16_t* out) {
  const dim3 g(grid_for(c.cap_pts, 4 * 64)), t(256);
  const auto args = [&](auto kern) {
    hipLaunchKernelGGL(kern, g, t, 0, c.stream, c.d_count, c.d_moff, b, b_lo, c.cap_model, code, c.hlast(),
                       c.w_head_plain, c.w_hbias, c.d_lse, out);
  };
  if (mode == TB_FREQ) args(k_table256r<C, TB_FREQ>);
  else if (mode == TB_CDF) args(k_table256r<C, TB_CDF>);
  else if (mode == TB_ENTRY) args(k_table256r<C, TB_ENTRY>);
  else args(k_table256r<C, TB_IV>);
}

template <int C>
void run_table16r(Ctx& c, int mode, int stage, int b, int b_lo, const uint8_t* code, uint16_t* out) {
  const dim3 g(grid_for(c.cap_pts, 16 * 64)), t(256);
  const auto args = [&](auto kern) {
    hipLaunchKernelGGL(kern, g, t, 0, c.stream, c.d_count, c.d_moff, b, b_lo, c.cap_model, code, c.hlast(),
                       c.w_head_plain, c.w_hbias, c.w_emb, c.d_s1, c.d_lse, c.d_lse2, out);
  };
  if (mode == TB_IV) args(k_table16r<C, TB_IV, 0>);
  else if (mode == TB_FREQ) stage == 1 ? args(k_table16r<C, TB_FREQ, 1>) : args(k_table16r<C, TB_FREQ, 2>);
  else if (mode == TB_ENTRY) stage == 1 ? args(k_table16r<C, TB_ENTRY, 1>) : args(k_table16r<C, TB_ENTRY, 2>);
  else stage == 1 ? args(k_table16r<C, TB_CDF, 1>) : args(k_table16r<C, TB_CDF, 2>);
}

bool table_regs(const Ctx& c) { return c.p.channels == 16 || c.p.channels == 32; }

void run_table(Ctx& c, bool sixteen, int mode, int stage, int b, int b_lo, const uint8_t* code, uint16_t* out) {
  if (sixteen)
    c.p.channels == 32 ? run_table16r<32>(c, mode, stage, b, b_lo, code, out)
                       : run_table16r<16>(c, mode, stage, b, b_lo, code, out);
  else
    c.p.channels == 32 ? run_table256r<32>(c, mode, b, b_lo, code, out)
                       : run_table256r<16>(c, mode, b, b_lo, code, out);
}

hipError_t launch_symbol_freqs(Ctx& c, int b, uint16_t* freq) {
  ProfScope ps_(c, RENO_K_OTHER);
  if (table_regs(c)) {
    run_table(c, false, TB_FREQ, 0, b, b, nullptr, freq);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_symbol_freqs, dim3(grid_for(c.cap_pts, 4)), dim3(256), 0, c.stream,
                     c.d_count, c.d_moff, b, c.cap_model, c.hlast(), c.p.channels, c.w_head_plain,
                     c.w_hbias, c.d_lse, freq);
  return hipGetLastError();
}

hipError_t launch_symbol_freqs16(Ctx& c, int b, int stage, uint16_t* freq) {
  ProfScope ps_(c, RENO_K_OTHER);
  if (table_regs(c)) {
    run_table(c, true, TB_FREQ, stage, b, b, nullptr, freq);
    return hipGetLastError();
  }
  hipLaunchKernelGGL(k_symbol_freqs16, dim3(grid_for(c.cap_pts, 16)), dim3(256), 0, c.stream,
                     c.d_count, c.d_moff, b, stage, c.cap_model, c.hlast(), c.p.channels, c.w_head_plain,
                     c.w_hbias, c.w_emb, c.d_s1, c.d_lse, c.d_lse2, freq);
  return hipGetLastError();
}

hipError_t launch_symbol_cdf(Ctx& c, int b, int stage, uint16_t* start) {
  ProfScope ps_(c, RENO_K_OTHER);
  if (table_regs(c)) {
    run_table(c, stage != 0, TB_CDF, stage, b, b, nullptr, start);
    return hipGetLastError();
  }
  if (stage == 0)
    hipLaunchKernelGGL(k_symbol_cdf, dim3(grid_for(c.cap_pts, 4)), dim3(256), 0, c.stream,
                       c.d_count, c.d_moff, b, c.cap_model, c.hlast(), c.p.channels, c.w_head_plain,
                       c.w_hbias, c.d_lse, start);
  else
    hipLaunchKernelGGL(k_symbol_cdf16, dim3(grid_for(c.cap_pts, 16)), dim3(256), 0, c.stream,
                       c.d_count, c.d_moff, b, stage, c.cap_model, c.hlast(), c.p.channels, c.w_head_plain,
                       c.w_hbias, c.w_emb, c.d_s1, c.d_lse, c.d_lse2, start);
  return hipGetLastError();
}

hipError_t launch_symbol_entries(Ctx& c, int b, int stage, uint32_t* entries, uint16_t* scratch) {
  if (table_regs(c)) {
    ProfScope ps_(c, RENO_K_OTHER);
    run_table(c, stage != 0, TB_ENTRY, stage, b, b, nullptr, reinterpret_cast<uint16_t*>(entries));
    return hipGetLastError();
  }
  hipError_t e = launch_symbol_cdf(c, b, stage, scratch);
  if (e != hipSuccess) return e;
  ProfScope ps_(c, RENO_K_OTHER);
  const int K = stage == 0 ? 256 : 16;
  hipLaunchKernelGGL(k_cdf_entries, dim3(grid_for(c.cap_pts * K, 256)), dim3(256), 0, c.stream, c.d_count, b, K,
                     scratch, entries);
  return hipGetLastError();
}

hipError_t launch_symbol_intervals(Ctx& c, int b_lo, int b_hi, uint16_t* iv) {
  ProfScope ps_(c, RENO_K_OTHER);
  const bool two = c.p.head_mode == RENO_HEAD_TWO_STAGE;
  // model rows of consecutive scales are consecutive, so each scale's output
  // starts at its model-row offset relative to b_lo (read on the device)
  for (int b = b_lo; b <= b_hi; ++b) {
    if (table_regs(c))
      run_table(c, two, TB_IV, 0, b, b_lo, c.lv_code + c.lv(b), iv);
    else if (two)
      hipLaunchKernelGGL(k_symbol_intervals16, dim3(grid_for(c.cap_pts, 16)), dim3(256), 0, c.stream,
                         c.d_count, c.d_moff, b, b_lo, c.cap_model, c.lv_code + c.lv(b), c.hlast(),
                         c.p.channels, c.w_head_plain, c.w_hbias, c.w_emb, c.d_lse, c.d_lse2, iv);
    else
      hipLaunchKernelGGL(k_symbol_intervals, dim3(grid_for(c.cap_pts, 4)), dim3(256), 0, c.stream,
                         c.d_count, c.d_moff, b, b_lo, c.cap_model, c.lv_code + c.lv(b), c.hlast(),
                         c.p.channels, c.w_head_plain, c.w_hbias, c.d_lse, iv);
  }
  return hipGetLastError();
}

hipError_t launch_coords(Ctx& c, int b, int32_t* xyz, uint64_t* keys) {
  ProfScope ps_(c, RENO_K_OTHER);
  hipLaunchKernelGGL(k_coords, dim3(grid_for(c.cap_pts, 256)), dim3(256), 0, c.stream,
                     c.lv_key + c.lv(b), c.d_count, b, xyz, keys);
  return hipGetLastError();
}

hipError_t launch_copy_level_u8(Ctx& c, int b, uint8_t* out) {
  ProfScope ps_(c, RENO_K_OTHER);
  hipLaunchKernelGGL(k_copy_u8, dim3(grid_for(c.cap_pts, 256)), dim3(256), 0, c.stream,
                     c.lv_code + c.lv(b), c.d_count, b, out);
  return hipGetLastError();
}

hipError_t launch_copy_level_i32(Ctx& c, int b, const int32_t* src, int32_t* out) {
  ProfScope ps_(c, RENO_K_OTHER);
  hipLaunchKernelGGL(k_copy_i32, dim3(grid_for(c.cap_pts, 256)), dim3(256), 0, c.stream, src,
                     c.d_count, b, 1, out);
  return hipGetLastError();
}

hipError_t launch_neighbor_map(Ctx& c, int b, int32_t* out) {
  ProfScope ps_(c, RENO_K_OTHER);
  const int kv = c.top() ? c.kvol() : 27;
  hipLaunchKernelGGL(k_copy_map, dim3(grid_for(c.cap_pts * kv, 256)), dim3(256), 0, c.stream,
                     c.d_nbr, c.d_moff, c.d_count, b, c.cap_model, kv, c.nbr_stride(), out);
  return hipGetLastError();
}

}  // namespace reno
