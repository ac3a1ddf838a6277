// Decoder side on gfx950: the initial state (C^0, O^0) of Eq. 2 and the FCG
// expansion of Sec. 3.1 (expand each code to 8 bits, keep the children whose
// bit is set), as a single-pass popcount scan with decoupled look-back.  The
// children of a scale come out in ascending Morton order, identical to the
// encoder's sorted scale, and are inserted into the coordinate hash.

#include <algorithm>
#include <mutex>

#include "ctx.h"

namespace reno {
namespace {

// Scale b0 from int32 xyz and codes, strictly ascending in (frame, Morton)
// order; a frame batch gives each voxel's frame id (key f << 3b0 | Morton).
struct BaseArgs {
  const int32_t* xyz;
  const int32_t* frame_of;  // null: one frame
  int frames;
  const uint8_t* codes;
  int64_t n;
  int b0;
  uint64_t* key;
  uint8_t* code;
  int32_t* parent;
  int32_t* count;
  int32_t* moff;
  uint64_t* hreg;
  int hash_lg;
  uint32_t* err;
};

// Thread i of the base scale: voxel i for i < n; i == n closes the hash
// region table of a frame batch.
__device__ __forceinline__ void set_base_voxel(const BaseArgs& a, int64_t i) {
  const int64_t n = a.n;
  const int b0 = a.b0;
  if (i == 0) {
    a.count[b0] = (int32_t)n;
    a.moff[b0 + 1] = 0;
  }
  // hash regions of a frame batch in proportion to each frame's base voxels:
  // the thread of the first voxel of a frame (ids ascending; out-of-range ids
  // clamped, they are latched below) writes the starts of the frames since
  // the previous voxel's frame
  if (a.frame_of && i <= n) {
    const uint64_t T = 1ull << a.hash_lg;
    auto fid = [&](int64_t j) {
      const int32_t f = a.frame_of[j];
      return f < 0 ? 0 : (f >= a.frames ? a.frames - 1 : f);
    };
    const int f_hi = i < n ? fid(i) : a.frames;          // frames f_lo+1 .. f_hi start at voxel i
    const int f_lo = i > 0 ? fid(i - 1) : -1;
    const uint64_t st = n > 0 ? (uint64_t)i * T / (uint64_t)n : 0ull;
    for (int f = f_lo + 1; f <= f_hi; ++f) a.hreg[f] = f == a.frames ? T : st;
  }
  if (i >= n) return;
  const int32_t lim = 1 << b0;
  uint32_t q[3], qp[3];
  bool range_ok = true;
  for (int ax = 0; ax < 3; ++ax) {
    const int32_t v = a.xyz[3 * i + ax];
    range_ok = range_ok && v >= 0 && v < lim;
    q[ax] = (uint32_t)v & (uint32_t)(lim - 1);
  }
  if (!range_ok) latch(a.err, ERR_BASE_RANGE);
  int32_t f = 0, fp = 0;
  if (a.frame_of) {
    f = a.frame_of[i];
    if (f < 0 || f >= a.frames) {
      latch(a.err, ERR_FRAMES);
      f = 0;
    }
    if (i > 0) {
      fp = a.frame_of[i - 1];
      fp = (fp < 0 || fp >= a.frames) ? 0 : fp;
    }
  }
  const uint64_t k = morton3(q[0], q[1], q[2]) | ((uint64_t)f << (3 * b0));
  if (i > 0) {
    for (int ax = 0; ax < 3; ++ax) qp[ax] = (uint32_t)a.xyz[3 * (i - 1) + ax] & (uint32_t)(lim - 1);
    if ((morton3(qp[0], qp[1], qp[2]) | ((uint64_t)fp << (3 * b0))) >= k) latch(a.err, ERR_BASE_ORDER);
  }
  const uint8_t c = a.codes[i];
  if (c == 0) latch(a.err, ERR_ZERO_CODE);
  a.key[i] = k;
  a.code[i] = c;
  a.parent[i] = -1;
}

__global__ void __launch_bounds__(256) k_set_base(BaseArgs a) {
  set_base_voxel(a, (int64_t)blockIdx.x * blockDim.x + threadIdx.x);
}

// A new decoder frame whose base scale fits one block (n < 256): the frame's
// clear and the base scale in one launch.  Every block zeroes its share of
// the large ranges; block 0 alone clears the error word, the scale counts and
// the row offsets and then, after a barrier, writes the base scale (which
// sets a count and an offset and may latch errors), so no other block touches
// a word that block 0 writes.
constexpr int BASE_ONE_BLOCK = 256;
struct ClearBaseArgs {
  uint4* p[8];        // ranges every block zeroes
  uint64_t n16[8];
  int n;
  uint4* s[CLEAR_SMALL];  // ranges block 0 zeroes before the base scale
  uint32_t s16[CLEAR_SMALL];
  BaseArgs base;
};

__global__ void __launch_bounds__(BASE_ONE_BLOCK) k_clear_set_base(ClearBaseArgs a) {
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  const uint64_t g = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  for (int r = 0; r < a.n; ++r) {
    uint4* p = a.p[r];
    const uint64_t n = a.n16[r];
    for (uint64_t i = g; i < n; i += stride) p[i] = make_uint4(0u, 0u, 0u, 0u);
  }
  if (blockIdx.x != 0) return;
  for (int r = 0; r < CLEAR_SMALL; ++r)
    for (uint32_t i = threadIdx.x; i < a.s16[r]; i += blockDim.x) a.s[r][i] = make_uint4(0u, 0u, 0u, 0u);
  __syncthreads();
  set_base_voxel(a.base, threadIdx.x);
}

struct ExpArgs {
  const uint8_t* codes_in;  // caller codes for O_b, or null (already recorded)
  int b, B;
  int fb;                   // frame-id bits above the Morton bits
  int64_t cap_pts;
  int64_t cap_model;
  const uint64_t* key_b;
  uint8_t* code_b;
  int32_t* fc_b;      // first-child row of each parent (or null)
  uint64_t* key_n;    // scale b+1
  int32_t* parent_n;
  uint16_t* feat_n;   // layer-1 input word of each child (or null)
  int32_t* count;
  int32_t* moff;
  uint32_t* status;
  uint32_t* ticket;
  HashSlot* hash;
  int hash_lg;
  const uint64_t* hreg;  // hash region starts of a frame batch (null: one frame)
  uint32_t* err;
  int check_keys;     // latch ERR_KEY_RANGE for parent keys of 2^61 or more
};

__global__ void __launch_bounds__(EXP_THREADS) k_expand(ExpArgs a) {
  __shared__ uint32_t s_tile;
  __shared__ uint32_t s_wtot[EXP_THREADS / 64];
  __shared__ uint32_t s_base;
  constexpr int NW = EXP_THREADS / 64;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int64_t np = a.count[a.b];
  const int64_t ntiles = (np + EXP_TILE - 1) / EXP_TILE;
  const int bn = a.b + 1;
  if (ntiles == 0) {
    if (blockIdx.x == 0 && tid == 0) {
      a.count[bn] = 0;
      if (bn < a.B) a.moff[bn + 1] = a.moff[bn];
    }
    return;
  }
  // The grid is sized for the largest scale.  Only the first ntiles blocks
  // take a ticket, so they get exactly tickets 0 .. ntiles-1; the others leave
  // without touching the counter (same-address atomics serialise, and a ticket
  // per idle block cost microseconds at the small scales).
  if ((int64_t)blockIdx.x >= ntiles) return;
  if (tid == 0) s_tile = atomicAdd(a.ticket, 1u);
  __syncthreads();
  const int64_t tile = s_tile;
  if (tile >= ntiles) return;
  const int64_t base = tile * EXP_TILE;

  // popcount scan over the tile's parents (element j of wave w: w*64*KPT + j*64 + lane)
  uint32_t code[EXP_KPT], incl[EXP_KPT];
  uint64_t key[EXP_KPT];  // loaded with the codes: off the look-back's critical path
  uint32_t run = 0;
#pragma unroll
  for (int j = 0; j < EXP_KPT; ++j) {
    const int64_t p = base + (int64_t)w * 64 * EXP_KPT + j * 64 + lane;
    uint32_t c = 0;
    key[j] = p < np ? a.key_b[p] : 0ull;
    if (p < np) {
      c = a.codes_in ? a.codes_in[p] : a.code_b[p];
      if (a.codes_in) a.code_b[p] = (uint8_t)c;
      if (c == 0u) latch(a.err, ERR_ZERO_CODE);
      if (a.check_keys && (key[j] >> 61)) latch(a.err, ERR_KEY_RANGE);
    }
    code[j] = c;
    uint32_t x = (uint32_t)__popc(c);
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)x, o);
      if (lane >= o) x += y;
    }
    incl[j] = run + x;
    run += (uint32_t)__shfl((int)x, 63);
  }
  if (lane == 0) s_wtot[w] = run;
  __syncthreads();
  if (w == 0) {
    uint32_t tot = 0;
    for (int i = 0; i < NW; ++i) tot += s_wtot[i];
    const uint32_t ex = lookback_wave(a.status, (int)tile, tot, a.err);
    if (lane == 0) {
      s_base = ex;
      uint32_t acc = 0;
      for (int i = 0; i < NW; ++i) {
        const uint32_t t = s_wtot[i];
        s_wtot[i] = acc;
        acc += t;
      }
      if (tile == ntiles - 1) {
        int64_t nn = (int64_t)ex + tot;
        if (nn > a.cap_pts) {
          latch(a.err, ERR_CAPACITY);
          nn = a.cap_pts;
        }
        a.count[bn] = (int32_t)nn;
        if (bn < a.B) {
          const int64_t mo = (int64_t)a.moff[bn] + nn;
          if (mo > a.cap_model) latch(a.err, ERR_CAPACITY);
          a.moff[bn + 1] = (int32_t)mo;
        }
      }
    }
  }
  __syncthreads();
  const int64_t wbase = (int64_t)s_base + s_wtot[w];
#pragma unroll
  for (int j = 0; j < EXP_KPT; ++j) {
    const int64_t p = base + (int64_t)w * 64 * EXP_KPT + j * 64 + lane;
    if (p >= np) continue;
    const uint32_t c = code[j];
    int64_t q = wbase + incl[j] - (uint32_t)__popc(c);
    if (a.fc_b) a.fc_b[p] = (int32_t)q;
    const uint64_t kp = key[j] << 3;
    for (uint32_t d = 0; d < 8; ++d) {
      if (!((c >> d) & 1u)) continue;
      if (q >= a.cap_pts) {
        latch(a.err, ERR_CAPACITY);
        break;
      }
      a.key_n[q] = kp | d;
      a.parent_n[q] = (int32_t)p;
      if (a.feat_n) a.feat_n[q] = (uint16_t)(d | (c << 3));
      ++q;
    }
  }
  // the parents (scale b) go into the coordinate hash with their code and
  // first child when scale b+1 is a model scale
  if (bn >= a.B) return;
#pragma unroll
  for (int j = 0; j < EXP_KPT; ++j) {
    const int64_t p = base + (int64_t)w * 64 * EXP_KPT + j * 64 + lane;
    if (p >= np) continue;
    const int64_t q = wbase + incl[j] - (uint32_t)__popc(code[j]);
    hash_insert(a.hash, a.hash_lg, hash_region(a.hreg, a.hash_lg, frame_part(key[j], a.b)),
                tag_key(key[j], a.b, a.fb), (int32_t)q, code[j], a.err);
  }
}

// ---- FCG expansion without a context and without allocation ----
// Scratch of reno_expand_noalloc, one copy per device for the life of the
// process: NA_HEAD header words (parent count, child count, tile ticket, error
// word) and one look-back status word per tile of EXP_TILE parents.  Host code
// reaches it only through the address hipGetSymbolAddress returns for the
// current device; calls that overlap on one device share it and race.
constexpr int NA_HEAD = 64;
constexpr int NA_COUNT = 0;   // int32 [2]: parents (scale "0"), children (scale "1")
constexpr int NA_TICKET = 2;
constexpr int NA_ERR = 3;
constexpr int64_t NA_TILES = RENO_NOALLOC_MAX_PARENTS / EXP_TILE;
static_assert(RENO_NOALLOC_MAX_PARENTS % EXP_TILE == 0, "whole tiles");
static __device__ __align__(256) uint32_t scratch[NA_HEAD + NA_TILES];

// Clears the header and the status words of the call's tiles (a fill kernel
// rather than a memset, so that the call can be captured into a graph) and
// records the parent count where k_expand reads it.
__global__ void __launch_bounds__(256) k_noalloc_begin(uint32_t* s, int64_t n, int64_t words) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < words;
       i += (int64_t)gridDim.x * blockDim.x)
    s[i] = i == NA_COUNT ? (uint32_t)n : 0u;
}

// Child count and status of the call: result[0] = children written (clamped
// to the capacity), result[1] = 0 or the reno_status of a data error.
__global__ void k_noalloc_end(const uint32_t* s, int64_t* result) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  const uint32_t e = s[NA_ERR];
  int64_t st = RENO_OK;
  if (e & ERR_CAPACITY)
    st = RENO_E_CAPACITY;
  else if (e & (ERR_ZERO_CODE | ERR_KEY_RANGE))
    st = RENO_E_INPUT;
  else if (e)
    st = RENO_E_HIP;   // a look-back wait ran out (never expected)
  result[0] = (int64_t)(int32_t)s[NA_COUNT + 1];
  result[1] = st;
}

std::mutex g_na_mu;
uint32_t* g_na_ptr[RENO_NOALLOC_MAX_DEVICES] = {};

}  // namespace

hipError_t noalloc_scratch(uint32_t** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= RENO_NOALLOC_MAX_DEVICES) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_na_mu);
  if (!g_na_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_na_ptr[dev] = static_cast<uint32_t*>(p);
  }
  *out = g_na_ptr[dev];
  return hipSuccess;
}

hipError_t launch_expand_noalloc(const uint64_t* keys, const uint8_t* codes, int64_t n,
                                 uint64_t* child_keys, int32_t* child_parent, int64_t cap_children,
                                 int32_t* first_child, int64_t* result, hipStream_t stream) {
  uint32_t* s = nullptr;
  hipError_t e = noalloc_scratch(&s);
  if (e != hipSuccess) return e;
  const int64_t ntiles = (n + EXP_TILE - 1) / EXP_TILE;
  const int64_t words = NA_HEAD + ntiles;
  hipLaunchKernelGGL(k_noalloc_begin, dim3((unsigned)std::min<int64_t>((words + 255) / 256, 1024)), dim3(256), 0, stream, s, n, words);
  ExpArgs a;
  a.codes_in = nullptr;                       // the codes are read, never written
  a.b = 0;                                    // count[0]: parents, count[1]: children
  a.B = 1;                                    // no next model scale: no hash inserts, no row offsets
  a.fb = 0;
  a.cap_pts = cap_children;
  a.cap_model = 0;
  a.key_b = keys;
  a.code_b = const_cast<uint8_t*>(codes);
  a.fc_b = first_child;
  a.key_n = child_keys;
  a.parent_n = child_parent;
  a.feat_n = nullptr;
  a.count = reinterpret_cast<int32_t*>(s + NA_COUNT);
  a.moff = nullptr;                           // only touched when b + 1 < B
  a.status = s + NA_HEAD;
  a.ticket = s + NA_TICKET;
  a.hash = nullptr;
  a.hash_lg = 0;
  a.hreg = nullptr;
  a.err = s + NA_ERR;
  a.check_keys = 1;
  hipLaunchKernelGGL(k_expand, dim3((unsigned)(ntiles > 0 ? ntiles : 1)), dim3(EXP_THREADS), 0, stream, a);
  hipLaunchKernelGGL(k_noalloc_end, dim3(1), dim3(64), 0, stream, s, result);
  return hipGetLastError();
}

BaseArgs base_args(Ctx& c, const int32_t* xyz, const int32_t* frame_of, const uint8_t* codes, int64_t n) {
  const int b0 = c.b0();
  return BaseArgs{xyz, frame_of, c.frames, codes, n, b0, c.lv_key + c.lv(b0), c.lv_code + c.lv(b0),
                  c.lv_parent + c.lv(b0), c.d_count, c.d_moff, c.d_hreg, c.hash_lg, c.d_err};
}

hipError_t launch_set_base(Ctx& c, const int32_t* xyz, const int32_t* frame_of, const uint8_t* codes, int64_t n,
                           int B) {
  ProfScope ps_(c, RENO_K_SET_BASE);
  (void)B;
  int64_t blocks = (n + 1 + 255) / 256;   // thread n closes the hash region table
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_set_base, dim3((unsigned)blocks), dim3(256), 0, c.stream,
                     base_args(c, xyz, frame_of, codes, n));
  return hipGetLastError();
}

bool clear_set_base_fits(int64_t n) { return n >= 0 && n < BASE_ONE_BLOCK; }

hipError_t launch_clear_set_base(Ctx& c, const int32_t* xyz, const int32_t* frame_of, const uint8_t* codes,
                                 int64_t n) {
  if (!clear_set_base_fits(n)) return hipErrorInvalidValue;
  ProfScope ps_(c, RENO_K_SET_BASE);
  void* ptr[8];
  size_t bytes[8];
  const int k = frame_clear(c, ptr, bytes);
  ClearBaseArgs a{};
  uint64_t most = 0;
  for (int i = 0; i < CLEAR_SMALL; ++i) {
    a.s[i] = static_cast<uint4*>(ptr[i]);
    a.s16[i] = (uint32_t)((bytes[i] + 15) / 16);
  }
  a.n = 0;
  for (int i = CLEAR_SMALL; i < k && a.n < 8; ++i, ++a.n) {
    a.p[a.n] = static_cast<uint4*>(ptr[i]);
    a.n16[a.n] = (bytes[i] + 15) / 16;
    if (a.n16[a.n] > most) most = a.n16[a.n];
  }
  a.base = base_args(c, xyz, frame_of, codes, n);
  uint64_t blocks = (most + BASE_ONE_BLOCK - 1) / BASE_ONE_BLOCK;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_clear_set_base, dim3((unsigned)blocks), dim3(BASE_ONE_BLOCK), 0, c.stream, a);
  return hipGetLastError();
}

hipError_t launch_expand(Ctx& c, int b, const uint8_t* codes, int B) {
  ProfScope ps_(c, RENO_K_EXPAND);
  ExpArgs a;
  a.codes_in = codes;
  a.b = b;
  a.B = B;
  a.fb = c.fbits;
  a.cap_pts = c.cap_pts;
  a.cap_model = c.cap_model;
  a.key_b = c.lv_key + c.lv(b);
  a.code_b = c.lv_code + c.lv(b);
  a.fc_b = c.lv_fc + c.lv(b);
  a.key_n = c.lv_key + c.lv(b + 1);
  a.parent_n = c.lv_parent + c.lv(b + 1);
  a.feat_n = c.lv_feat + c.lv(b + 1);
  a.count = c.d_count;
  a.moff = c.d_moff;
  const int64_t max_tiles = c.exp_tiles;
  a.status = c.st_exp(b);
  a.ticket = c.d_ticket + TK_EXPAND + b;
  a.hash = c.d_hash;
  a.hash_lg = c.hash_lg;
  a.hreg = c.hreg();
  a.err = c.d_err;
  a.check_keys = 0;                           // context keys hold at most 3 * 20 + 10 bits
  hipLaunchKernelGGL(k_expand, dim3((unsigned)max_tiles), dim3(EXP_THREADS), 0, c.stream, a);
  return hipGetLastError();
}

}  // namespace reno
