// Device-side helpers shared by the HIP kernels of the codec hot path:
// Morton bit spreading, error latching, wavefront primitives, the decoupled
// look-back used by every single-pass scan, and the open-addressing
// coordinate hash.  gfx950 (CDNA4) only: wave64, 64-bit ballots.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace reno {

// ---- error latch (ctx device word), reported by the next synchronising call ----
enum : uint32_t {
  ERR_NONFINITE = 1u,    // a non-finite input coordinate
  ERR_CAPACITY = 2u,     // a scale or the model batch exceeded the context capacity
  ERR_HASH_FULL = 4u,    // coordinate hash ran out of slots
  ERR_ZERO_CODE = 8u,    // a code of 0 given to the decoder (codes lie in [1, 255])
  ERR_BASE_ORDER = 16u,  // base voxels not strictly ascending
  ERR_BASE_RANGE = 32u,  // base voxel outside [0, 2^b0)
  ERR_SPIN = 64u,        // a look-back wait exceeded its bound (never expected)
  ERR_DUP_KEY = 128u,    // the same key inserted twice (never expected: keys are a set)
  ERR_INTERNAL = 256u,   // an internal consistency check failed (never expected)
  ERR_SYMBOL = 512u,     // a decoded sub-code outside its alphabet (S1 above 15)
  ERR_FRAMES = 1024u,    // frame ranges or base frame ids of a frame batch malformed
  ERR_KEY_RANGE = 2048u, // a parent key of 2^61 or more (its children would not fit in 64 bits)
  ERR_STREAM = 4096u,    // an entropy-coded section or stream of a frame bitstream malformed
};

__device__ __forceinline__ void latch(uint32_t* err, uint32_t bit) { atomicOr(err, bit); }

// ---- Morton keys: x bit i -> key bit 3i, y -> 3i+1, z -> 3i+2 (21 bits per axis) ----
__device__ __forceinline__ uint64_t spread3(uint64_t x) {
  x &= 0x1fffffull;
  x = (x | (x << 32)) & 0x001f00000000ffffull;
  x = (x | (x << 16)) & 0x001f0000ff0000ffull;
  x = (x | (x << 8)) & 0x100f00f00f00f00full;
  x = (x | (x << 4)) & 0x10c30c30c30c30c3ull;
  x = (x | (x << 2)) & 0x1249249249249249ull;
  return x;
}

__device__ __forceinline__ uint32_t compact3(uint64_t x) {
  x &= 0x1249249249249249ull;
  x = (x ^ (x >> 2)) & 0x10c30c30c30c30c3ull;
  x = (x ^ (x >> 4)) & 0x100f00f00f00f00full;
  x = (x ^ (x >> 8)) & 0x001f0000ff0000ffull;
  x = (x ^ (x >> 16)) & 0x001f00000000ffffull;
  x = (x ^ (x >> 32)) & 0x1fffffull;
  return (uint32_t)x;
}

__device__ __forceinline__ uint64_t morton3(uint32_t x, uint32_t y, uint32_t z) {
  return spread3(x) | (spread3(y) << 1) | (spread3(z) << 2);
}

// ---- wavefront primitives (wave64) ----
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

// number of set bits of `mask` below this lane
__device__ __forceinline__ uint32_t rank_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

__device__ __forceinline__ uint32_t wave_or(uint32_t v) {
  for (int o = 32; o > 0; o >>= 1) v |= (uint32_t)__shfl_xor((int)v, o);
  return v;
}

// ---- agent-scope relaxed atomics on look-back status words ----
__device__ __forceinline__ uint32_t ld_status(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_status(uint32_t* p, uint32_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Decoupled look-back (single-pass prefix over tiles processed in ticket
// order).  Status word = 2 flag bits | 30-bit count; 0 = not yet published.
constexpr uint32_t LB_AGG = 1u << 30;
constexpr uint32_t LB_INC = 2u << 30;
constexpr uint32_t LB_VAL = (1u << 30) - 1u;
constexpr uint32_t LB_SPIN_LIMIT = 1u << 24;

// The calling thread owns counter `c` of tile `tile` (status row stride
// `width`).  Publishes the tile aggregate, walks back over earlier tiles until
// an inclusive prefix is found, publishes its own inclusive prefix and returns
// the exclusive one.  The walk reads LB_BATCH predecessors per round trip and
// consumes them in order, stopping at the first inclusive prefix or retrying
// from the first one not yet published.  Earlier tiles took their tickets
// earlier and are therefore already running; each publishes its aggregate
// without waiting, so every wait ends.  A bound on the wait latches ERR_SPIN
// instead of hanging.
constexpr int LB_BATCH = 8;

// An inclusive prefix beyond the 30-bit field (only reachable with corrupt
// decoder codes on a context of more than 2^27 points) would spill into the
// flag bits; it is published saturated and latches ERR_CAPACITY instead, so
// the capacity checks downstream see a count above any context capacity.
__device__ __forceinline__ uint32_t lb_saturate(uint32_t v, uint32_t* err) {
  if (v > LB_VAL) {
    latch(err, ERR_CAPACITY);
    return LB_VAL;
  }
  return v;
}

__device__ __forceinline__ uint32_t lookback(uint32_t* status, int width, int tile, int c,
                                             uint32_t agg, uint32_t* err) {
  uint32_t* mine = status + (size_t)tile * width + c;
  if (tile == 0) {
    st_status(mine, LB_INC | agg);
    return 0;
  }
  st_status(mine, LB_AGG | agg);
  uint32_t excl = 0;
  uint32_t spins = 0;
  for (int t = tile - 1; t >= 0;) {
    uint32_t v[LB_BATCH];
#pragma unroll
    for (int i = 0; i < LB_BATCH; ++i)
      v[i] = (t - i >= 0) ? ld_status(status + (size_t)(t - i) * width + c) : LB_INC;
    int used = 0;
    bool done = false, wait = false;
#pragma unroll
    for (int i = 0; i < LB_BATCH; ++i) {
      if (done || wait) continue;
      const uint32_t f = v[i] & ~LB_VAL;
      if (f == 0) {
        wait = true;
        continue;
      }
      excl += v[i] & LB_VAL;
      ++used;
      if (f == LB_INC) done = true;
    }
    if (done) break;
    t -= used;
    if (wait) {
      if (++spins > LB_SPIN_LIMIT) {
        latch(err, ERR_SPIN);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  st_status(mine, LB_INC | lb_saturate(excl + agg, err));
  return excl;
}

// Single-counter look-back run by all 64 lanes of one wavefront: lane i reads
// predecessor t-i, so one round trip covers 64 tiles.  Returns the exclusive
// prefix (same value in every lane).
__device__ __forceinline__ uint32_t lookback_wave(uint32_t* status, int tile, uint32_t agg,
                                                  uint32_t* err) {
  const int lane = (int)(threadIdx.x & 63);
  if (tile == 0) {
    if (lane == 0) st_status(status, LB_INC | agg);
    return 0;
  }
  if (lane == 0) st_status(status + tile, LB_AGG | agg);
  uint32_t excl = 0;
  uint32_t spins = 0;
  for (int t = tile - 1; t >= 0;) {
    const int my = t - lane;
    const uint32_t v = my >= 0 ? ld_status(status + my) : LB_INC;
    const uint32_t f = v & ~LB_VAL;
    const uint64_t notready = __ballot(f == 0);
    const uint64_t inc = __ballot(f == LB_INC);
    const uint64_t stop = notready | inc;
    // lanes before the first stopping lane hold aggregates to consume; an
    // inclusive prefix there ends the walk, an unpublished one is retried
    const int first = stop ? __builtin_ctzll(stop) : 64;
    const bool take_inc = first < 64 && ((inc >> first) & 1ull);
    const int ntake = first + (take_inc ? 1 : 0);
    uint32_t x = lane < ntake ? (v & LB_VAL) : 0u;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += (uint32_t)__shfl_xor((int)x, o);
    excl += x;
    if (take_inc) break;
    t -= ntake;
    if (first < 64) {  // a predecessor has not published yet
      if (++spins > LB_SPIN_LIMIT) {
        latch(err, ERR_SPIN);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
  }
  if (lane == 0) st_status(status + tile, LB_INC | lb_saturate(excl + agg, err));
  return excl;
}

// ---- open-addressing coordinate hash in HBM ----
// Maps a voxel of a parent scale to its occupancy code and the row of its
// first child, so that any cell of the next scale can be resolved from one
// probe: the child with octant d exists iff bit d of the code is set, and its
// row is first + popcount(code & ((1 << d) - 1)) (the FCG order).  One table
// serves every scale of a frame (or of a batch of frames): a scale-b key is
// tagged with a sentinel bit at position 3b + fb, where fb is the number of
// frame-id bits kept above the 3b Morton bits (0 for a single frame; key <
// 2^{3b + fb}), which makes tagged keys of different scales distinct and
// never 0 (0 marks an empty slot).
struct alignas(16) HashSlot {
  unsigned long long key;
  int32_t first;   // row of the first child in the next scale
  uint32_t code;   // occupancy code of the voxel
};

__device__ __forceinline__ uint64_t tag_key(uint64_t key, int b, int fb) { return key | (1ull << (3 * b + fb)); }

// A scale-b key of a frame batch: frame id above the 3b Morton bits, so the
// parent of a key is key >> 3 and keys sort by (frame, Morton order).
__device__ __forceinline__ uint64_t morton_part(uint64_t key, int b) {
  return b >= 21 ? key : key & ((1ull << (3 * b)) - 1ull);
}
__device__ __forceinline__ uint64_t frame_part(uint64_t key, int b) { return b >= 21 ? 0ull : key >> (3 * b); }

// Home slots of a frame: a frame batch gives each frame its own region
// [base, base + size) of the table (sized by the frame's share of the batch),
// so that the inserts and probes of the frames in flight stay within a few
// regions instead of the whole table; probing still runs on linearly through
// the whole table, so a region that fills up spills into the next one.  A
// single frame's region is the whole table.
struct HashReg {
  uint64_t base, size;
};

// Region of frame f from the table of region starts (null: one frame).
__device__ __forceinline__ HashReg hash_region(const uint64_t* reg, int lg, uint64_t f) {
  if (!reg) return HashReg{0ull, 1ull << lg};
  return HashReg{reg[f], reg[f + 1] - reg[f]};
}

// Multiplicative hash scaled to the region: base + floor(mix * size / 2^64)
// (for the whole table, the top lg bits of the product).
__device__ __forceinline__ uint32_t hash_home(uint64_t tk, const HashReg& r) {
  return (uint32_t)(r.base + __umul64hi(tk * 0x9E3779B97F4A7C15ull, r.size));
}

// Inserts tagged key -> (first, code) with linear probing (64-bit CAS on the key).
__device__ __forceinline__ void hash_insert(HashSlot* tab, int lg, const HashReg& reg, uint64_t tk,
                                            int32_t first, uint32_t code, uint32_t* err) {
  const uint32_t mask = (1u << lg) - 1u;
  uint32_t h = hash_home(tk, reg) & mask;
  for (uint32_t step = 0; step <= mask; ++step) {
    unsigned long long prev = atomicCAS(&tab[h].key, 0ull, (unsigned long long)tk);
    if (prev == 0ull) {
      tab[h].first = first;
      tab[h].code = code;
      return;
    }
    if (prev == tk) {
      latch(err, ERR_DUP_KEY);
      return;
    }
    h = (h + 1u) & mask;
  }
  latch(err, ERR_HASH_FULL);
}

// (first, code) of a tagged key; code 0 (no children) when absent.  The
// table was built by an earlier kernel.
__device__ __forceinline__ uint2 hash_find(const HashSlot* tab, int lg, const HashReg& reg, uint64_t tk) {
  const uint32_t mask = (1u << lg) - 1u;
  uint32_t h = hash_home(tk, reg) & mask;
  for (uint32_t step = 0; step <= mask; ++step) {
    const uint4 s = *reinterpret_cast<const uint4*>(&tab[h]);
    const uint64_t k = ((uint64_t)s.y << 32) | s.x;
    if (k == tk) return make_uint2(s.z, s.w);
    if (k == 0ull) return make_uint2(0u, 0u);
    h = (h + 1u) & mask;
  }
  return make_uint2(0u, 0u);
}

// N lookups at once, all of one frame (tk == 0: no query, result code 0): the
// home slots of all queries are loaded together, so a lane pays one memory
// round trip unless a query lands on a slot holding another key.
template <int N>
__device__ __forceinline__ void hash_find_n(const HashSlot* tab, int lg, const HashReg& reg, const uint64_t* tk,
                                            uint2* out) {
  const uint32_t mask = (1u << lg) - 1u;
  uint4 s[N];
#pragma unroll
  for (int j = 0; j < N; ++j)
    s[j] = *reinterpret_cast<const uint4*>(&tab[hash_home(tk[j] ? tk[j] : 1ull, reg) & mask]);
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const uint64_t k = ((uint64_t)s[j].y << 32) | s[j].x;
    out[j] = make_uint2(0u, 0u);
    if (!tk[j]) continue;
    if (k == tk[j])
      out[j] = make_uint2(s[j].z, s[j].w);
    else if (k != 0ull)  // collision: continue linear probing from the home slot
      out[j] = hash_find(tab, lg, reg, tk[j]);
  }
}

}  // namespace reno
