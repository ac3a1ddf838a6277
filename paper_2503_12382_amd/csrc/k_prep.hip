// Encoder front end on gfx950: quantisation to the B-bit grid, Morton keys,
// LSD radix sort (single pass per digit with decoupled look-back), the
// multiscale pyramid by dyadic downscaling (Sec. 3, Eq. 1) and the FOG
// occupancy codes (Sec. 3.1).
//
// Quantisation is bit-exact with a plain CPU evaluation: fp64, no
// contraction, correctly rounded division, floor and clamp.

#include "ctx.h"

#pragma clang fp contract(off)

namespace reno {
namespace {

// ---------------------------------------------------------------------------
// Zero-fill of up to 8 ranges (16-byte multiples) in one launch.  Used at the
// start of a frame for counters, histograms, look-back status and the hash.
struct ZeroArgs {
  uint4* p[8];
  uint64_t n16[8];
  int n;
};

__global__ void __launch_bounds__(256) k_zero(ZeroArgs a) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int r = 0; r < a.n; ++r) {
    uint4* p = a.p[r];
    const uint64_t n = a.n16[r];
    for (uint64_t i = g; i < n; i += stride) p[i] = make_uint4(0u, 0u, 0u, 0u);
  }
}

// ---------------------------------------------------------------------------
// Histogram update of every sort pass's digit of key k in LDS, aggregated over
// runs of adjacent lanes with equal digits: one LDS atomic per run.  Input
// points arrive in scan order, so the coarse digits of neighbouring lanes
// mostly agree (unaggregated, those atomics would hit one address and
// serialise), while the fine digits differ and cost one atomic per lane, as
// without aggregation.
__device__ __forceinline__ void digit_count(uint32_t dig, bool valid, uint32_t* h) {
  const int lane = lane_id();
  const uint32_t prev = (uint32_t)__shfl_up((int)dig, 1);
  const uint64_t valids = __ballot(valid);
  const bool vprev = lane > 0 && ((valids >> (lane - 1)) & 1ull);
  const bool head = valid && (!vprev || prev != dig);
  const uint64_t heads = __ballot(head);
  if (head) {
    const uint64_t above = lane == 63 ? 0ull : (heads >> (lane + 1)) << (lane + 1);
    const uint64_t upto = above ? (above & (0ull - above)) - 1ull : ~0ull;  // lanes below the next head
    const uint64_t run = valids & upto & ~((1ull << lane) - 1ull);
    atomicAdd(&h[dig], (uint32_t)__popcll(run));
  }
}

__device__ __forceinline__ void digits_of(uint64_t k, int passes, uint32_t* sh) {
  for (int ps = 0; ps < passes; ++ps)
    digit_count((uint32_t)(k >> (RADIX_BITS * ps)) & (RADIX - 1), true, sh + ps * RADIX);
}

__device__ __forceinline__ void digits_of_idle(int passes, uint32_t* sh) {
  for (int ps = 0; ps < passes; ++ps) digit_count(0u, false, sh + ps * RADIX);
}

// ---------------------------------------------------------------------------
// Quantise + Morton + digit histograms of every sort pass.
//   u = ((p + R) * 2^B) / (2R) in fp64, q = clamp(floor(u), 0, 2^B - 1).
//   Frame batch: point i of frame f (frame_start[f] <= i < frame_start[f+1])
//   gets the key f << 3B | Morton(q).
__global__ void __launch_bounds__(256) k_quantize(const float* __restrict__ pts, int64_t n, int B,
                                                  double R, const int64_t* __restrict__ frame_start,
                                                  int frames, uint64_t* __restrict__ keys,
                                                  uint32_t* __restrict__ hist, int passes,
                                                  uint64_t* __restrict__ hreg, int hash_lg,
                                                  uint32_t* err) {
  __shared__ uint32_t sh[MAX_PASSES * RADIX];
  __shared__ int64_t s_fs[RENO_MAX_FRAMES + 1];  // frame ranges of a batch
  for (int i = threadIdx.x; i < passes * RADIX; i += blockDim.x) sh[i] = 0u;
  if (frames > 1) {
    for (int f = threadIdx.x; f <= frames; f += blockDim.x) s_fs[f] = frame_start[f];
    if (blockIdx.x == 0 && threadIdx.x == 0) {  // 0 = s_0 <= s_1 <= ... <= s_F = n
      bool ok = frame_start[0] == 0 && frame_start[frames] == n;
      for (int f = 0; f < frames; ++f) ok = ok && frame_start[f] <= frame_start[f + 1];
      if (!ok) latch(err, ERR_FRAMES);
    }
    // hash region of each frame in proportion to its points (region starts
    // ascending from 0 to the table size even for malformed ranges)
    if (blockIdx.x == 0) {
      const uint64_t T = 1ull << hash_lg;
      for (int f = threadIdx.x; f <= frames; f += blockDim.x) {
        int64_t sf = f == frames ? n : frame_start[f];
        sf = sf < 0 ? 0 : (sf > n ? n : sf);
        uint64_t st = n > 0 ? (uint64_t)sf * T / (uint64_t)n : (uint64_t)f * T / (uint64_t)frames;
        if (f == frames) st = T;
        hreg[f] = st;
      }
    }
  }
  __syncthreads();
  int fcur = 0;  // a thread's points increase, so its frame only moves forward
  const double scale = (double)(int64_t(1) << B);
  const double span = 2.0 * R;
  const double top = (double)((int64_t(1) << B) - 1);
  bool bad = false;
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // QU points per thread per iteration, all loads issued first.  Every lane
  // of a wave runs the same number of iterations so that the wave-wide digit
  // matching below sees all lanes; idle lanes carry no key.
  constexpr int QU = 4;
  const int64_t nwaves_iter = (n + stride * QU - 1) / (stride * QU);
  for (int64_t it = 0; it < nwaves_iter; ++it) {
    float pv[QU][3];
#pragma unroll
    for (int u = 0; u < QU; ++u) {
      const int64_t i = (it * QU + u) * stride + gid;
#pragma unroll
      for (int a = 0; a < 3; ++a) pv[u][a] = i < n ? pts[3 * i + a] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < QU; ++u) {
      const int64_t i = (it * QU + u) * stride + gid;
      if (i >= n) {
        digits_of_idle(passes, sh);
        continue;
      }
      uint32_t q[3];
#pragma unroll
      for (int a = 0; a < 3; ++a) {
        const float p = pv[u][a];
        if (!isfinite(p)) {
          bad = true;
          q[a] = 0u;
          continue;
        }
        const double uu = ((double)p + R) * scale / span;
        double f = floor(uu);
        f = f < 0.0 ? 0.0 : f;
        f = f > top ? top : f;
        q[a] = (uint32_t)f;
      }
      uint64_t k = morton3(q[0], q[1], q[2]);
      if (frames > 1) {  // last frame f with s_fs[f] <= i
        while (fcur + 1 < frames && s_fs[fcur + 1] <= i) ++fcur;
        k |= (uint64_t)fcur << (3 * B);
      }
      keys[i] = k;
      digits_of(k, passes, sh);
    }
  }
  if (bad) latch(err, ERR_NONFINITE);
  __syncthreads();
  for (int i = threadIdx.x; i < passes * RADIX; i += blockDim.x)
    if (sh[i]) atomicAdd(&hist[i], sh[i]);
}

// Exclusive scan of one value per thread over a 256-thread block.
__device__ __forceinline__ uint32_t block_excl_scan256(uint32_t v, uint32_t* s_wsum) {
  const int lane = lane_id(), w = threadIdx.x >> 6;
  uint32_t x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = (uint32_t)__shfl_up((int)x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) s_wsum[w] = x;
  __syncthreads();
  uint32_t off = 0;
  for (int i = 0; i < w; ++i) off += s_wsum[i];
  __syncthreads();
  return off + x - v;
}

// ---------------------------------------------------------------------------
// One LSD radix-sort pass over 8-bit digit `pass` (stable).  Tiles are taken
// in ticket order; each tile ranks its keys with wave-level digit matching,
// publishes per-digit counts, finds its global offsets by look-back, reorders
// in LDS and writes out bucket runs.
template <int KPT>
__global__ void __launch_bounds__(SORT_THREADS) k_sort_pass(const uint64_t* __restrict__ in,
                                                            uint64_t* __restrict__ out, int64_t n,
                                                            int shift,
                                                            const uint32_t* __restrict__ hist,
                                                            uint32_t* status, uint32_t* ticket,
                                                            uint32_t* err) {
  constexpr int TILE = SORT_THREADS * KPT;
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_wh[4][RADIX];
  __shared__ uint32_t s_dexcl[RADIX];
  __shared__ uint32_t s_gbase[RADIX];
  __shared__ uint32_t s_wsum[4];
  __shared__ uint64_t s_keys[TILE];

  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  if (tid == 0) s_tile = atomicAdd(ticket, 1u);
  for (int i = tid; i < 4 * RADIX; i += SORT_THREADS) (&s_wh[0][0])[i] = 0u;
  __syncthreads();
  const int tile = (int)s_tile;
  const int64_t base = (int64_t)tile * TILE;

  uint64_t key[KPT];
  uint32_t dig[KPT], rnk[KPT];
  bool ok[KPT];
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    const int64_t idx = base + (int64_t)w * 64 * KPT + j * 64 + lane;
    ok[j] = idx < n;
    key[j] = ok[j] ? in[idx] : 0ull;
    dig[j] = (uint32_t)(key[j] >> shift) & (RADIX - 1);
  }
#pragma unroll
  for (int j = 0; j < KPT; ++j) {
    uint64_t peers = __ballot(ok[j]);
#pragma unroll
    for (int bit = 0; bit < RADIX_BITS; ++bit) {
      const bool set = (dig[j] >> bit) & 1u;
      const uint64_t bm = __ballot(set);
      peers &= set ? bm : ~bm;
    }
    // the leader lane updates the count that every lane of the group has just
    // read; volatile keeps the compiler from reusing a value across slots
    volatile uint32_t* cnt = &s_wh[w][dig[j]];
    const uint32_t below = rank_below(peers);
    const uint32_t before = *cnt;
    if (ok[j] && below == 0u) *cnt = before + (uint32_t)__popcll(peers);
    rnk[j] = before + below;
  }
  __syncthreads();

  // digit t = tid: per-wave exclusive offsets, tile count, global base
  const int d = tid;
  const uint32_t c0 = s_wh[0][d], c1 = s_wh[1][d], c2 = s_wh[2][d], c3 = s_wh[3][d];
  const uint32_t tot = c0 + c1 + c2 + c3;
  s_wh[0][d] = 0u;
  s_wh[1][d] = c0;
  s_wh[2][d] = c0 + c1;
  s_wh[3][d] = c0 + c1 + c2;
  const uint32_t dex = block_excl_scan256(tot, s_wsum);
  s_dexcl[d] = dex;
  const uint32_t gex = block_excl_scan256(hist[d], s_wsum);
  const uint32_t prev = lookback(status, RADIX, tile, d, tot, err);
  s_gbase[d] = gex + prev;
  __syncthreads();

#pragma unroll
  for (int j = 0; j < KPT; ++j)
    if (ok[j]) s_keys[s_dexcl[dig[j]] + s_wh[w][dig[j]] + rnk[j]] = key[j];
  __syncthreads();

  const int cnt = (int)((n - base) < TILE ? (n - base) : TILE);
  for (int q = tid; q < cnt; q += SORT_THREADS) {
    const uint64_t k = s_keys[q];
    const uint32_t dd = (uint32_t)(k >> shift) & (RADIX - 1);
    out[s_gbase[dd] + (uint32_t)q - s_dexcl[dd]] = k;
  }
}

// ---------------------------------------------------------------------------
// Pyramid: from the sorted finest keys S[0..n) (duplicates allowed) build every
// scale b0..B at once.  Element i is the first element of its run at scale b
// iff lv(i) <= b - b0, where lv(i) = max(0, B - floor(h/3) - b0), h = highest
// bit of S[i] ^ S[i-1] (lv(0) = 0; duplicates never start a run).  Its row in
// V_b is the number of such elements before it, found with per-scale ballots
// and a look-back over tiles.  Also writes parent rows and first-child rows.
struct PyrArgs {
  const uint64_t* S;
  int64_t n;
  int B, b0, nl;
  int64_t cap_pts;
  int64_t cap_model;
  uint64_t* key;
  int32_t* parent;
  int32_t* fc;
  int32_t* count;
  int32_t* moff;
  uint32_t* status;
  uint32_t* ticket;
  HashSlot* hash;
  int hash_lg;
  uint32_t* err;
};

__global__ void __launch_bounds__(PYR_THREADS) k_pyramid(PyrArgs a) {
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_wc[4][NLEV];     // per-wave counts -> exclusive offsets
  __shared__ uint32_t s_gb[NLEV];        // global exclusive base of the tile per scale
  __shared__ uint32_t s_tot[NLEV];       // inclusive totals (last tile)
  __shared__ uint32_t s_jex[4][PYR_KPT][NLEV];  // per wave: elements before slot j
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int nl = a.nl;
  if (tid == 0) s_tile = atomicAdd(a.ticket, 1u);
  __syncthreads();
  const int tile = (int)s_tile;
  const int64_t base = (int64_t)tile * PYR_TILE;

  int lvj[PYR_KPT];
  uint64_t kj[PYR_KPT];
#pragma unroll
  for (int j = 0; j < PYR_KPT; ++j) {
    const int64_t i = base + (int64_t)w * 64 * PYR_KPT + j * 64 + lane;
    int lv = nl;  // absent
    uint64_t k = 0;
    if (i < a.n) {
      k = a.S[i];
      if (i == 0) {
        lv = 0;
      } else {
        const uint64_t x = k ^ a.S[i - 1];
        if (x != 0ull) {
          const int h = 63 - __clzll((long long)x);
          const int l = a.B - h / 3 - a.b0;
          lv = l < 0 ? 0 : l;
        }
      }
    }
    lvj[j] = lv;
    kj[j] = k;
  }
  // phase 1: per-wave counts per scale, and per element slot j (read-only in
  // phase 2, so no lane ever depends on another lane's LDS update)
  for (int l = 0; l < nl; ++l) {
    uint32_t c = 0;
#pragma unroll
    for (int j = 0; j < PYR_KPT; ++j) {
      if (lane == 0) s_jex[w][j][l] = c;
      c += (uint32_t)__popcll(__ballot(lvj[j] <= l));
    }
    if (lane == 0) s_wc[w][l] = c;
  }
  __syncthreads();
  if (tid < nl) {
    const int l = tid;
    const uint32_t c0 = s_wc[0][l], c1 = s_wc[1][l], c2 = s_wc[2][l], c3 = s_wc[3][l];
    s_wc[0][l] = 0u;
    s_wc[1][l] = c0;
    s_wc[2][l] = c0 + c1;
    s_wc[3][l] = c0 + c1 + c2;
    const uint32_t tot = c0 + c1 + c2 + c3;
    const uint32_t ex = lookback(a.status, NLEV, tile, l, tot, a.err);
    s_gb[l] = ex;
    s_tot[l] = ex + tot;
  }
  __syncthreads();
  // phase 2: ranks and writes; row at scale l = tile base + wave offset +
  // earlier slots of the wave + lanes below in this slot
#pragma unroll
  for (int j = 0; j < PYR_KPT; ++j) {
    const int lv = lvj[j];
    int32_t prev_pos = -1;  // exclusive count at scale l-1
    for (int l = 0; l < nl; ++l) {
      const bool here = lv <= l;
      const uint64_t m = __ballot(here);
      const uint32_t pos = s_gb[l] + s_wc[w][l] + s_jex[w][j][l] + rank_below(m);
      if (here) {
        const int b = a.b0 + l;
        const int64_t r = (int64_t)l * a.cap_pts + pos;
        const uint64_t kb = kj[j] >> (3 * (a.B - b));
        a.key[r] = kb;
        // parent: at the element's coarsest scale the representative of its
        // parent run precedes it (exclusive count - 1); above, it is itself
        a.parent[r] = (l == 0) ? -1 : (l == lv ? prev_pos - 1 : prev_pos);
        if (l > lv) a.fc[(int64_t)(l - 1) * a.cap_pts + prev_pos] = (int32_t)pos;
      }
      prev_pos = (int32_t)pos;
    }
  }
  // last tile: publish N_b and the packed model offsets
  if (tile == (int)((a.n + PYR_TILE - 1) / PYR_TILE) - 1 && tid == 0) {
    int64_t acc = 0;
    for (int l = 0; l < nl; ++l) {
      const int b = a.b0 + l;
      a.count[b] = (int32_t)s_tot[l];
      if (b > a.b0) {
        a.moff[b] = (int32_t)acc;
        if (b < a.B) acc += s_tot[l];
      }
    }
    if (acc > a.cap_model) latch(a.err, ERR_CAPACITY);
  }
}

// ---------------------------------------------------------------------------
// FOG codes for every scale b0 <= b < B: the children of parent p are the
// rows [fc[p], fc[p+1]) of V_{b+1}; the code ORs 1 << (child key & 7)
// (Sec. 3.1: weights 1..128 over the octants).  Also writes each child's
// layer-1 input bits (delta | code << 3) and inserts every parent of a model
// scale (b0 <= b <= B-2) into the coordinate hash with its code and first child.
__global__ void __launch_bounds__(256) k_codes(const uint64_t* __restrict__ key,
                                               const int32_t* __restrict__ fc,
                                               uint8_t* __restrict__ code,
                                               uint16_t* __restrict__ feat,
                                               const int32_t* __restrict__ count, int b0, int B,
                                               int64_t cap_pts, HashSlot* hash, int hash_lg,
                                               const uint64_t* __restrict__ hreg, int fb, uint32_t* err) {
  __shared__ int64_t s_pre[NLEV + 1];
  if (threadIdx.x == 0) {
    int64_t acc = 0;
    for (int b = b0; b < B; ++b) {
      s_pre[b - b0] = acc;
      acc += count[b];
    }
    s_pre[B - b0] = acc;
  }
  __syncthreads();
  const int nl = B - b0;
  const int64_t total = s_pre[nl];
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += stride) {
    int l = 0;
    while (l + 1 < nl && s_pre[l + 1] <= t) ++l;
    const int b = b0 + l;
    const int64_t p = t - s_pre[l];
    const int64_t np = count[b];
    const int64_t rb = (int64_t)l * cap_pts, rc = (int64_t)(l + 1) * cap_pts;
    const int32_t nn = count[b + 1];
    const int32_t lo = fc[rb + p];
    const int32_t hi = (p + 1 < np) ? fc[rb + p + 1] : nn;
    if (lo < 0 || hi > nn || hi <= lo || hi - lo > 8) {  // never expected: children runs are 1..8
      latch(err, ERR_INTERNAL);
      continue;
    }
    const int nk = hi - lo;
    // all child keys are loaded at once (clamped rows), then used from registers
    uint64_t kc[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) kc[i] = key[rc + lo + (i < nk ? i : nk - 1)];
    uint32_t c = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i < nk) c |= 1u << (uint32_t)(kc[i] & 7ull);
    code[rb + p] = (uint8_t)c;
#pragma unroll
    for (int i = 0; i < 8; ++i)
      if (i < nk) feat[rc + lo + i] = (uint16_t)((kc[i] & 7ull) | (c << 3));
    // parents of model scales go into the coordinate hash with their code
    // and first child
    if (b <= B - 2) {
      const uint64_t kp = key[rb + p];
      hash_insert(hash, hash_lg, hash_region(hreg, hash_lg, frame_part(kp, b)), tag_key(kp, b, fb), lo, c, err);
    }
  }
}

}  // namespace

hipError_t launch_zero(Ctx& c, void* const* ptrs, const size_t* bytes, int n) {
  ProfScope ps_(c, RENO_K_ZERO);
  ZeroArgs a{};
  uint64_t most = 0;
  for (int i = 0; i < n && i < 8; ++i) {
    a.p[i] = static_cast<uint4*>(ptrs[i]);
    a.n16[i] = (bytes[i] + 15) / 16;
    if (a.n16[i] > most) most = a.n16[i];
  }
  a.n = n < 8 ? n : 8;
  uint64_t blocks = (most + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_zero, dim3((unsigned)blocks), dim3(256), 0, c.stream, a);
  return hipGetLastError();
}

hipError_t launch_quantize(Ctx& c, const float* pts, int64_t n, int B, int passes, const int64_t* frame_start,
                           int frames) {
  ProfScope ps_(c, RENO_K_QUANTIZE);
  int64_t blocks = (n + 1023) / 1024;  // 4 points per thread per iteration
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_quantize, dim3((unsigned)blocks), dim3(256), 0, c.stream, pts, n, B,
                     c.p.range_m, frame_start, frames, c.keys_a, c.d_hist, passes, c.d_hreg, c.hash_lg,
                     c.d_err);
  return hipGetLastError();
}

hipError_t launch_sort_pass(Ctx& c, const uint64_t* in, uint64_t* out, int64_t n, int pass) {
  ProfScope ps_(c, RENO_K_SORT);
  uint32_t* status = c.st_sort(pass);
  // large inputs: 4096-key tiles (digit runs of ~16 keys per tile, a quarter
  // of the look-backs); small ones keep 1024-key tiles to fill the CUs
  if (n >= SORT_BIG_N) {
    const int64_t tiles = (n + SORT_THREADS * SORT_KPT_BIG - 1) / (SORT_THREADS * SORT_KPT_BIG);
    hipLaunchKernelGGL(k_sort_pass<SORT_KPT_BIG>, dim3((unsigned)tiles), dim3(SORT_THREADS), 0, c.stream, in, out,
                       n, RADIX_BITS * pass, c.d_hist + pass * RADIX, status, c.d_ticket + TK_SORT + pass, c.d_err);
  } else {
    const int64_t tiles = (n + SORT_TILE - 1) / SORT_TILE;
    hipLaunchKernelGGL(k_sort_pass<SORT_KPT>, dim3((unsigned)tiles), dim3(SORT_THREADS), 0, c.stream, in, out,
                       n, RADIX_BITS * pass, c.d_hist + pass * RADIX, status, c.d_ticket + TK_SORT + pass, c.d_err);
  }
  return hipGetLastError();
}

hipError_t launch_pyramid(Ctx& c, const uint64_t* sorted, int64_t n, int B) {
  ProfScope ps_(c, RENO_K_PYRAMID);
  PyrArgs a;
  a.S = sorted;
  a.n = n;
  a.B = B;
  a.b0 = c.b0();
  a.nl = B - c.b0() + 1;
  a.cap_pts = c.cap_pts;
  a.cap_model = c.cap_model;
  a.key = c.lv_key;
  a.parent = c.lv_parent;
  a.fc = c.lv_fc;
  a.count = c.d_count;
  a.moff = c.d_moff;
  a.status = c.st_pyr();
  a.ticket = c.d_ticket + TK_PYR;
  a.hash = c.d_hash;
  a.hash_lg = c.hash_lg;
  a.err = c.d_err;
  const int64_t tiles = (n + PYR_TILE - 1) / PYR_TILE;
  hipLaunchKernelGGL(k_pyramid, dim3((unsigned)tiles), dim3(PYR_THREADS), 0, c.stream, a);
  return hipGetLastError();
}

hipError_t launch_codes(Ctx& c, int B) {
  ProfScope ps_(c, RENO_K_CODES);
  int64_t work = (int64_t)(B - c.b0()) * c.npoints;
  int64_t blocks = (work + 255) / 256;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_codes, dim3((unsigned)blocks), dim3(256), 0, c.stream, c.lv_key, c.lv_fc,
                     c.lv_code, c.lv_feat, c.d_count, c.b0(), B, c.cap_pts, c.d_hash, c.hash_lg,
                     c.hreg(), c.fbits, c.d_err);
  return hipGetLastError();
}

}  // namespace reno
