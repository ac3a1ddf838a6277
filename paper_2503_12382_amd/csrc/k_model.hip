// Target occupancy predictor (Sec. 3.2, Eq. 5) on gfx950, in the configured
// form: per voxel of a scale, the 11 input bits [delta, parent code] (target
// embedding, Eqs. 7-8), L submanifold 3x3x3 sparse conv + ReLU layers on the
// target coordinates (Eq. 9) and a linear head to 256 logits with the softmax
// normaliser (Eq. 10).
//
// Work unit: a wavefront owns a tile of 16 consecutive voxels of one scale.
// Each layer is computed transposed, out^T[c_out][16] = sum_k W_k^T in_k^T, on
// fp32 MFMA 16x16x4: the A operand is the offset's weights (staged once per
// block in LDS, pre-swizzled so each lane reads its operands with 128-bit
// loads), the B operand is the gathered neighbour rows (each lane loads a
// contiguous slice of one neighbour row).  Only offsets with at least one
// occupied neighbour in the tile are issued.  The accumulator layout of the
// last conv layer is exactly the B operand layout of the head, so the head
// (16 x 256 logits per tile) runs from registers, followed by a row max / sum
// of exp over the 64 logits a lane holds and the 4 lanes sharing a voxel.
// Output-stationary: no atomics, a fixed summation order per voxel, so an
// encoder and a decoder evaluating the same scale get bit-identical results.

#include "ctx.h"

namespace reno {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int CONV_THREADS = 512;
constexpr int CONV_WAVES = CONV_THREADS / 64;
constexpr int KCH = 4;  // offsets whose gathers are in flight together

__device__ __forceinline__ f4 mfma4(float a, float b, f4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// ---------------------------------------------------------------------------
// Weight packing.  Conv layer (C_in -> C): KS = ceil(C_in/4) MFMA k-steps per
// offset; lane l (g = l/16) feeds input channel ci = g*KS + s at step s and
// output channel co = 16*cb + l%16.  Packed [27][C/16][64][KSP], KSP = KS
// rounded up to 4, zero padded.
__global__ void k_pack_conv(const float* __restrict__ W, int c_in, int C, int KS, int KSP,
                            float* __restrict__ out) {
  const int ncb = C / 16;
  const int total = 27 * ncb * 64 * KSP;
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

// Head: step t = 4*cb + r carries channel c = 16*cb + 4*g + r (the conv
// accumulator register r of column block cb); lane l carries symbol
// 16*sb + l%16.  Packed [16][64][C/4].
__global__ void k_pack_head(const float* __restrict__ H, int C, float* __restrict__ out) {
  const int KT = C / 4;
  const int total = 16 * 64 * KT;
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
    const int t = i % KT;
    const int lane = (i / KT) % 64;
    const int sb = i / (KT * 64);
    const int c = 16 * (t >> 2) + 4 * (lane >> 4) + (t & 3);
    out[i] = H[(size_t)c * 256 + sb * 16 + (lane & 15)];
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
  int32_t* nbr;           // [cap_model][27]
  const float* h_in;      // [cap_model][C_in] (unused by the first layer)
  float* h_out;           // [cap_model][C]
  const float* w;         // packed conv weights
  const float* bias;      // [C]
  const float* hw;        // packed head weights (last layer)
  const float* hb;        // [256]
  float* lse;             // [cap_model]
  float* logits;          // optional [rows][256], row = packed row - moff[b_lo]
  uint32_t* err;
};

template <int C, bool FIRST, bool LAST>
__global__ void __launch_bounds__(CONV_THREADS) k_conv(ConvArgs a) {
  constexpr int NCB = C / 16;
  constexpr int KS = FIRST ? 3 : C / 4;
  constexpr int KSP = (KS + 3) & ~3;
  constexpr int KT = C / 4;
  constexpr int WSZ = 27 * NCB * 64 * KSP;
  constexpr int HSZ = LAST ? 16 * 64 * KT : 4;
  __shared__ __attribute__((aligned(16))) float s_w[WSZ];
  __shared__ __attribute__((aligned(16))) float s_h[HSZ];
  __shared__ int32_t s_map[CONV_WAVES][16 * 28];
  __shared__ int64_t s_tpre[NLEV + 1];

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int r = lane & 15, g = lane >> 4;
  const int nsc = a.b_hi - a.b_lo + 1;

  // tile prefix over the scales of this launch
  int64_t total_tiles = 0;
  for (int i = 0; i < nsc; ++i) {
    const int b = a.b_lo + i;
    int64_t nb = a.count[b];
    const int64_t mo = a.moff[b];
    if (mo + nb > a.cap_model) nb = 0;  // overflow was latched where the size was made
    total_tiles += (nb + 15) / 16;
  }
  const int64_t first_tile = (int64_t)blockIdx.x * CONV_WAVES;
  if (first_tile >= total_tiles) return;  // whole block idle: skip the weight staging
  if (tid == 0) {
    int64_t acc = 0;
    for (int i = 0; i < nsc; ++i) {
      const int b = a.b_lo + i;
      int64_t nb = a.count[b];
      if (a.moff[b] + nb > a.cap_model) nb = 0;
      s_tpre[i] = acc;
      acc += (nb + 15) / 16;
    }
    s_tpre[nsc] = acc;
  }
  // stage the weights (and head weights) in LDS
  {
    const f4* src = reinterpret_cast<const f4*>(a.w);
    f4* dst = reinterpret_cast<f4*>(s_w);
    for (int i = tid; i < WSZ / 4; i += CONV_THREADS) dst[i] = src[i];
    if (LAST) {
      const f4* hs = reinterpret_cast<const f4*>(a.hw);
      f4* hd = reinterpret_cast<f4*>(s_h);
      for (int i = tid; i < HSZ / 4; i += CONV_THREADS) hd[i] = hs[i];
    }
  }
  __syncthreads();

  const int64_t wave_stride = (int64_t)gridDim.x * CONV_WAVES;
  for (int64_t tile = first_tile + w; tile < total_tiles; tile += wave_stride) {
    int si = 0;
    while (si + 1 < nsc && s_tpre[si + 1] <= tile) ++si;
    const int b = a.b_lo + si;
    const int64_t nvox = a.count[b];
    const int64_t mo = a.moff[b];
    const int64_t row0 = (tile - s_tpre[si]) * 16;
    const int64_t row = row0 + r;
    const bool valid = row < nvox;
    const int64_t prow = mo + row;
    const int64_t lvb = (int64_t)(b - a.b0) * a.cap_pts;
    int32_t* map = s_map[w];

    // ---- neighbour rows of the tile: probe the hash (first layer) or load the map
    uint32_t present = 0;
    if (FIRST) {
      const uint64_t key = valid ? a.lv_key[lvb + row] : 0ull;
      const int x = (int)compact3(key), y = (int)compact3(key >> 1), z = (int)compact3(key >> 2);
      const int lim = 1 << b;
#pragma unroll
      for (int j = 0; j < 7; ++j) {
        const int k = 7 * g + j;
        if (k >= 27) break;
        int32_t nbv = -1;
        if (valid) {
          if (k == 13) {
            nbv = (int32_t)row;
          } else {
            const int xx = x + (k % 3) - 1, yy = y + (k / 3) % 3 - 1, zz = z + k / 9 - 1;
            if (xx >= 0 && yy >= 0 && zz >= 0 && xx < lim && yy < lim && zz < lim)
              nbv = hash_find(a.hash, a.hash_lg,
                              tag_key(morton3((uint32_t)xx, (uint32_t)yy, (uint32_t)zz), b));
          }
          a.nbr[prow * 27 + k] = nbv;
        }
        map[r * 28 + k] = nbv;
        present |= (nbv >= 0 ? 1u : 0u) << k;
      }
    } else {
#pragma unroll
      for (int j = 0; j < 7; ++j) {
        const int k = 7 * g + j;
        if (k >= 27) break;
        const int32_t nbv = valid ? a.nbr[prow * 27 + k] : -1;
        map[r * 28 + k] = nbv;
        present |= (nbv >= 0 ? 1u : 0u) << k;
      }
    }
    uint32_t offs = (uint32_t)__builtin_amdgcn_readfirstlane((int)wave_or(present));

    // ---- accumulate over the occupied offsets
    f4 acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      acc[cb] = *reinterpret_cast<const f4*>(a.bias + 16 * cb + 4 * g);
    }
    while (offs) {
      int ks[KCH];
#pragma unroll
      for (int c = 0; c < KCH; ++c) {
        ks[c] = offs ? __builtin_ctz(offs) : -1;
        offs &= offs ? offs - 1u : 0u;
      }
      float bsrc[KCH][KSP];
#pragma unroll
      for (int c = 0; c < KCH; ++c) {
        if (ks[c] < 0) break;
        const int32_t n = map[r * 28 + ks[c]];
        if (FIRST) {
          const uint32_t word = n >= 0 ? (uint32_t)a.lv_feat[lvb + n] : 0u;
#pragma unroll
          for (int s = 0; s < KSP; ++s) bsrc[c][s] = (float)((word >> (g * KS + s)) & 1u);
          // the fourth slot (s = 3) is padding and its weights are zero
        } else {
          if (n >= 0) {
            const f4* src = reinterpret_cast<const f4*>(a.h_in + (mo + n) * C + g * KS);
#pragma unroll
            for (int q = 0; q < KSP / 4; ++q) {
              const f4 v = src[q];
              bsrc[c][4 * q + 0] = v[0];
              bsrc[c][4 * q + 1] = v[1];
              bsrc[c][4 * q + 2] = v[2];
              bsrc[c][4 * q + 3] = v[3];
            }
          } else {
#pragma unroll
            for (int s = 0; s < KSP; ++s) bsrc[c][s] = 0.0f;
          }
        }
      }
#pragma unroll
      for (int c = 0; c < KCH; ++c) {
        if (ks[c] < 0) break;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const f4* wp = reinterpret_cast<const f4*>(s_w + ((ks[c] * NCB + cb) * 64 + lane) * KSP);
#pragma unroll
          for (int q = 0; q < KSP / 4; ++q) {
            const f4 wv = wp[q];
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (4 * q + e < KS) acc[cb] = mfma4(wv[e], bsrc[c][4 * q + e], acc[cb]);
          }
        }
      }
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int e = 0; e < 4; ++e) acc[cb][e] = fmaxf(acc[cb][e], 0.0f);
    if (valid) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
        *reinterpret_cast<f4*>(a.h_out + prow * C + 16 * cb + 4 * g) = acc[cb];
    }

    if (LAST) {
      // ---- head: z^T[256][16] = H^T h^T, B operand = the conv accumulators
      f4 zz[16];
#pragma unroll
      for (int sb = 0; sb < 16; ++sb) {
        zz[sb] = *reinterpret_cast<const f4*>(a.hb + 16 * sb + 4 * g);
        const f4* hp = reinterpret_cast<const f4*>(s_h + (sb * 64 + lane) * KT);
#pragma unroll
        for (int q = 0; q < KT / 4; ++q) {
          const f4 hv = hp[q];
#pragma unroll
          for (int e = 0; e < 4; ++e) zz[sb] = mfma4(hv[e], acc[q][e], zz[sb]);
        }
      }
      // lane holds symbols 16*sb + 4*g + e of voxel r; the 4 lanes r, r+16,
      // r+32, r+48 together hold all 256
      float m = zz[0][0];
#pragma unroll
      for (int sb = 0; sb < 16; ++sb)
#pragma unroll
        for (int e = 0; e < 4; ++e) m = fmaxf(m, zz[sb][e]);
      m = fmaxf(m, __shfl_xor(m, 16));
      m = fmaxf(m, __shfl_xor(m, 32));
      float s = 0.0f;
#pragma unroll
      for (int sb = 0; sb < 16; ++sb)
#pragma unroll
        for (int e = 0; e < 4; ++e) s += __expf(zz[sb][e] - m);
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      if (valid && g == 0) a.lse[prow] = m + __logf(s);
      if (a.logits && valid) {
        float* lo = a.logits + (prow - a.moff[a.b_lo]) * 256 + 4 * g;
#pragma unroll
        for (int sb = 0; sb < 16; ++sb) *reinterpret_cast<f4*>(lo + 16 * sb) = zz[sb];
      }
    }
  }
}

template <int C, bool FIRST, bool LAST>
hipError_t run_conv(Ctx& c, const ConvArgs& a) {
  // one block per CU is enough to stage the weights once and keep 8 waves busy
  hipLaunchKernelGGL((k_conv<C, FIRST, LAST>), dim3(256), dim3(CONV_THREADS), 0, c.stream, a);
  return hipGetLastError();
}

template <int C>
hipError_t run_layer(Ctx& c, bool first, bool last, const ConvArgs& a) {
  if (first && last) return run_conv<C, true, true>(c, a);
  if (first) return run_conv<C, true, false>(c, a);
  if (last) return run_conv<C, false, true>(c, a);
  return run_conv<C, false, false>(c, a);
}

}  // namespace

hipError_t launch_pack_weights(Ctx& c, const reno_weights& w) {
  ProfScope ps_(c, RENO_K_OTHER);
  const int C = c.p.channels;
  int c_in = RENO_IN_FEATURES;
  for (int l = 0; l < c.p.layers; ++l) {
    const int KS = (c_in + 3) / 4;
    const int KSP = (KS + 3) & ~3;
    hipLaunchKernelGGL(k_pack_conv, dim3(64), dim3(256), 0, c.stream, w.conv_w[l], c_in, C, KS, KSP,
                       c.w_conv[l]);
    hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(256), 0, c.stream, w.conv_b[l], c.w_bias[l], C);
    c_in = C;
  }
  hipLaunchKernelGGL(k_pack_head, dim3(32), dim3(256), 0, c.stream, w.head_w, C, c.w_head);
  hipLaunchKernelGGL(k_copy_f32, dim3(1), dim3(256), 0, c.stream, w.head_b, c.w_hbias, 256);
  hipLaunchKernelGGL(k_copy_f32, dim3(32), dim3(256), 0, c.stream, w.head_w, c.w_head_plain,
                     C * 256);
  return hipGetLastError();
}

hipError_t launch_model(Ctx& c, int b_lo, int b_hi, float* logits) {
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
  a.nbr = c.d_nbr;
  a.hb = c.w_hbias;
  a.hw = c.w_head;
  a.lse = c.d_lse;
  a.err = c.d_err;
  const int L = c.p.layers;
  hipError_t e = hipSuccess;
  for (int l = 0; l < L && e == hipSuccess; ++l) {
    a.h_in = (l & 1) ? c.h_a : c.h_b;   // layer l reads what layer l-1 wrote
    a.h_out = (l & 1) ? c.h_b : c.h_a;  // layer 0 writes h_a
    a.w = c.w_conv[l];
    a.bias = c.w_bias[l];
    a.logits = (l == L - 1) ? logits : nullptr;
    const bool first = l == 0, last = l == L - 1;
    ProfScope ps_(c, last ? RENO_K_CONV_LAST : (first ? RENO_K_CONV_FIRST : RENO_K_CONV_MID));
    e = (c.p.channels == 32) ? run_layer<32>(c, first, last, a) : run_layer<16>(c, first, last, a);
  }
  return e;
}

}  // namespace reno
