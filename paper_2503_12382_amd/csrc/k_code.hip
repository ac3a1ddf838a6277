// GPU entropy coder of the whole-frame bitstream (the arithmetic-coding step
// of Sec. 4.2, realised as rANS: Duda, arXiv:1311.2540).  State of 64 bits in
// [2^31, 2^63), 32-bit renormalisation words, 16-bit probability resolution.
// Each model scale, and each stage of the two-stage head, is one section of
// S = ceil(N / L) interleaved streams (symbol i goes to stream i mod S; L is
// the stream length in symbols, a parameter of the bitstream); every stream is
// the plain single-stream code of its symbols.
//
// Encoder: one thread per stream pushes its symbols' (start, freq) intervals
// in reverse, writing renormalisation words backwards into a private region;
// one workgroup then lays the streams out (a scan of their lengths), and a
// copy kernel moves them into place and bit-packs the base voxels.
// Decoder: one wavefront per stream.  The cumulative table of the next symbol
// sits across the 64 lanes (4 entries each); a ballot of "first entry <=
// slot" names the lane holding the symbol, whose entries are then read out
// and searched in scalar registers.  Tables do not depend on the coder
// state, so they are loaded several symbols ahead.

#include <type_traits>

#include "ctx.h"
#include "dev.h"

namespace reno {
namespace {

constexpr uint64_t kLow = 1ull << 31;  // lower end of the state interval
constexpr int kProb = 16;              // probability resolution (tables sum to 2^16)
constexpr int kRing = 32;              // decoder: symbols whose tables are in flight (divides 64)
constexpr int kDecWaves = 4;           // decoder: wavefronts (streams) per workgroup
constexpr int kLayThreads = 1024;

__device__ __forceinline__ int64_t streams_of(int64_t n, int L) { return n > 0 ? (n + L - 1) / L : 1; }

// Section t and stream j of global stream index g (sections in bitstream
// order: scale b_lo first, stages inner); false past the last stream.
__device__ bool locate(const int32_t* count, int b_lo, int sections, int stages, int L, int64_t g, int* t,
                       int64_t* j, int64_t* S) {
  int64_t acc = 0;
  for (int u = 0; u < sections; ++u) {
    const int64_t s = streams_of(count[b_lo + u / stages], L);
    if (g < acc + s) {
      *t = u;
      *j = g - acc;
      *S = s;
      return true;
    }
    acc += s;
  }
  return false;
}

struct EncArgs {
  const uint32_t* iv;    // (start | freq << 16) per voxel and stage: [model rows][stages]
  const int32_t* count;  // N_b
  const int32_t* moff;   // first model row of scale b
  int64_t cap_model;
  int b_lo, sections, stages, L;
  uint32_t* region;  // [G][L + 2], stream g written backwards from its end
  uint32_t* lens;    // [G] words of stream g
  int64_t G;
  uint32_t* err;
};

__device__ __forceinline__ uint32_t rfl(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }
__device__ __forceinline__ uint32_t rdl(uint32_t v, int lane) {
  return (uint32_t)__builtin_amdgcn_readlane((int)v, lane);
}

// v into lane `at` of a register whose other lanes keep old (at uniform)
__device__ __forceinline__ uint32_t wrl(uint32_t old, uint32_t v, int at) {
  return (int)(threadIdx.x & 63) == at ? v : old;
}

// Division by a symbol frequency 2 <= f < 2^16 for states x < 2^63 as a
// multiplication (Granlund and Montgomery, PLDI 1994, Thm. 4.2 with N = 63):
// with l = ceil(log2 f) and m = ceil(2^(63 + l) / f) < 2^64,
// floor(x / f) = floor(x m / 2^64) >> (l - 1).  m is computed by long
// division of 2^(63 + l) in 32-bit digits; each digit's quotient (dividend
// below 2^48) comes from a double division and is corrected by its remainder.
__device__ __forceinline__ uint32_t div48(uint64_t t, uint32_t f, uint32_t* r) {
  int64_t q = (int64_t)((double)t / (double)f);
  int64_t rm = (int64_t)t - q * (int64_t)f;
  if (rm < 0) {
    --q;
    rm += f;
  } else if (rm >= (int64_t)f) {
    ++q;
    rm -= f;
  }
  *r = (uint32_t)rm;
  return (uint32_t)q;
}

__device__ __forceinline__ uint64_t recip_magic(uint32_t f) {
  const int l = 32 - __clz(f - 1);           // ceil(log2 f), f >= 2
  uint32_t r;
  const uint32_t q1 = div48((uint64_t)1 << (31 + l), f, &r);  // 2^(l-1) * 2^32: the digit above is 0
  const uint32_t q0 = div48((uint64_t)r << 32, f, &r);
  return (((uint64_t)q1 << 32) | q0) + (r != 0);
}

// One wavefront per stream, its symbols pushed last to first in trips of 64:
// at the start of a trip lane u loads the interval of the trip's step u and
// prepares its division (multiplier and shift); the steps then read those
// through lane reads, so the coder state stays in scalar registers and its
// chain holds no memory access and no division.  Renormalisation words are
// collected in a register (lane e for the e-th word of the window) and
// written out 64 at a time, backwards from the end of the stream's region.
constexpr int kEncWaves = 4;

__global__ void __launch_bounds__(64 * kEncWaves) k_rans_encode(EncArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t g = (int64_t)blockIdx.x * kEncWaves + (int64_t)rfl(threadIdx.x >> 6);
  if (g >= a.G) return;
  int t;
  int64_t j, S;
  if (!locate(a.count, a.b_lo, a.sections, a.stages, a.L, g, &t, &j, &S)) return;
  const int b = a.b_lo + t / a.stages, s = t % a.stages;
  const int64_t row0 = (int64_t)a.moff[b] - a.moff[a.b_lo];
  int64_t n = a.count[b];
  if (a.moff[b] + n > a.cap_model) n = 0;  // overflow, latched where the size was made
  const int64_t m = n > j ? (n - j + S - 1) / S : 0;
  uint32_t* out = a.region + g * (int64_t)(a.L + 2);
  const uint32_t* iv = a.iv + (row0 + j) * a.stages + s;  // symbol k at iv[k * step]
  const int64_t step = S * a.stages;
  uint64_t x = kLow;
  int64_t w = a.L + 2;  // words of the region still free (the stream ends at the region's end)
  uint32_t win = 0;     // renormalisation words not yet written, lane e = e-th of them
  int nwin = 0;
  bool bad = false;
  auto emit = [&](uint32_t word) {
    win = wrl(win, word, nwin);
    if (++nwin == 64) {  // a full window: 64 words, the first emitted at the highest address
      out[w - 1 - lane] = win;
      w -= 64;
      nwin = 0;
    }
  };
  // lane u: the interval of step k0 + u (symbol m - 1 - k0 - u); the next
  // trip's are loaded at the start of a trip, so their latency is hidden
  auto trip_iv = [&](int64_t k0) { return iv[(k0 + lane < m ? m - 1 - k0 - lane : 0) * step]; };
  uint32_t iv_next = m > 0 ? trip_iv(0) : 0u;
  for (int64_t k0 = 0; k0 < m; k0 += 64) {
    const uint32_t iv_l = iv_next;
    const uint32_t f_l = iv_l >> 16;
    const uint64_t mg = f_l >= 2 ? recip_magic(f_l) : 0ull;
    const uint32_t mg_lo = (uint32_t)mg, mg_hi = (uint32_t)(mg >> 32);
    if (k0 + 64 < m) iv_next = trip_iv(k0 + 64);  // after this trip's values are in use
    const int nt = (int)(m - k0 < 64 ? m - k0 : 64);
    for (int u = 0; u < nt; ++u) {
      const uint32_t sf = rdl(iv_l, u);
      const uint32_t st = sf & 0xFFFFu, f = sf >> 16;
      const uint64_t mu = ((uint64_t)rdl(mg_hi, u) << 32) | rdl(mg_lo, u);
      if (f == 0) {  // the head kernels never produce an empty interval
        bad = true;
        continue;
      }
      // keep the state below 2^63 after the step: x / f < 2^(63 - 16)
      if ((uint32_t)(x >> 47) >= f) {  // x < 2^63: the quotient fits 16 bits
        emit((uint32_t)x);
        x >>= 32;
      }
      uint64_t q;
      if (f == 1) {
        q = x;
      } else {
        const int l = 32 - __clz(f - 1);
        q = __umul64hi(x, mu) >> (l - 1);
      }
      x = (q << kProb) + (x - q * f) + st;
    }
  }
  emit((uint32_t)x);  // final state: low word, then high word (first in decoding order)
  emit((uint32_t)(x >> 32));
  if (lane < nwin) out[w - 1 - lane] = win;
  w -= nwin;
  if (lane == 0) {
    a.lens[g] = (uint32_t)(a.L + 2 - w);
    if (bad) latch(a.err, ERR_INTERNAL);
  }
}

struct LayArgs {
  const int32_t* count;
  int b_lo, sections, stages, L, b0, B;
  const uint32_t* lens;
  int64_t G;
  int64_t* offs;  // [G] first word of stream g in the bitstream
  uint32_t* out;
  int64_t cap_words;
  int64_t* total;  // [0] bitstream words, [1] streams in use
  uint32_t* err;
};

// Bitstream layout: header (6 words), base voxels, then per section the
// stream lengths as 16-bit fields (two per word, stream 2q in the low half)
// followed by the streams.  One workgroup scans the streams' word counts.
__global__ void __launch_bounds__(kLayThreads) k_rans_layout(LayArgs a) {
  constexpr int MS = 2 * NLEV;
  __shared__ int64_t sec_first[MS + 1], sec_streams[MS], sec_start[MS];
  __shared__ int64_t part[kLayThreads];
  const int tid = threadIdx.x;
  if (tid == 0) {
    int64_t acc = 0;
    for (int u = 0; u < a.sections; ++u) {
      sec_first[u] = acc;
      sec_streams[u] = streams_of(a.count[a.b_lo + u / a.stages], a.L);
      acc += sec_streams[u];
    }
    sec_first[a.sections] = acc;
  }
  __syncthreads();
  const int64_t Gt = sec_first[a.sections];
  if (Gt > a.G) {  // the launch bound covers every stream
    if (tid == 0) latch(a.err, ERR_INTERNAL);
    return;
  }
  const int64_t n0 = a.count[a.b0];
  const int64_t base = 6 + (n0 * (3 * a.b0 + 8) + 31) / 32;
  const int64_t chunk = (Gt + kLayThreads - 1) / kLayThreads;
  const int64_t lo = (int64_t)tid * chunk, hi = min(Gt, lo + chunk);
  // words contributed by stream g: its own, plus its section's length words
  // when it is the section's first stream
  int64_t sum = 0;
  int u = 0;
  for (int64_t g = lo; g < hi; ++g) {
    while (g >= sec_first[u + 1]) ++u;
    sum += a.lens[g] + (g == sec_first[u] ? (sec_streams[u] + 1) / 2 : 0);
  }
  part[tid] = sum;
  __syncthreads();
  for (int d = 1; d < kLayThreads; d <<= 1) {
    const int64_t v = tid >= d ? part[tid - d] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int64_t pos = base + part[tid] - sum;
  u = 0;
  for (int64_t g = lo; g < hi; ++g) {
    while (g >= sec_first[u + 1]) ++u;
    if (g == sec_first[u]) {
      sec_start[u] = pos;
      pos += (sec_streams[u] + 1) / 2;
    }
    a.offs[g] = pos;
    pos += a.lens[g];
  }
  __syncthreads();
  u = 0;
  for (int64_t g = lo; g < hi; ++g) {
    while (g >= sec_first[u + 1]) ++u;
    const int64_t j = g - sec_first[u];
    if (j & 1) continue;
    const uint32_t word = a.lens[g] | (j + 1 < sec_streams[u] ? a.lens[g + 1] << 16 : 0u);
    const int64_t at = sec_start[u] + j / 2;
    if (at < a.cap_words) a.out[at] = word;
  }
  if (tid == 0) {
    const int64_t total = base + part[kLayThreads - 1];
    const uint32_t hdr[6] = {0x4F4E4552u, (uint32_t)a.B, (uint32_t)a.b0, (uint32_t)a.stages, (uint32_t)a.L,
                             (uint32_t)n0};
    for (int k = 0; k < 6; ++k) a.out[k] = hdr[k];
    a.total[0] = total;
    a.total[1] = Gt;
    if (total > a.cap_words) latch(a.err, ERR_INTERNAL);
  }
}

struct PackArgs {
  const uint32_t* region;
  const uint32_t* lens;
  const int64_t* offs;
  const int64_t* total;
  int L;
  int64_t G;
  const int32_t* xyz;   // [N_b0][3] base voxels
  const uint8_t* code;  // [N_b0] their codes
  const int32_t* count;
  int b0;
  uint32_t* out;
  int64_t cap_words;
};

// Blocks below G: stream g to its place; the rest: base-voxel words (word q
// takes the bits 32q .. 32q + 31 of the fields x | y << b0 | z << 2b0 |
// code << 3b0, each 3 b0 + 8 bits wide, packed from the lowest bit up).
__global__ void __launch_bounds__(256) k_rans_pack(PackArgs a) {
  if ((int64_t)blockIdx.x < a.G) {
    const int64_t g = blockIdx.x;
    if (g >= a.total[1]) return;
    const int64_t len = a.lens[g], dst = a.offs[g];
    const uint32_t* src = a.region + g * (int64_t)(a.L + 2) + (a.L + 2 - len);
    for (int64_t w = threadIdx.x; w < len; w += 256)
      if (dst + w < a.cap_words) a.out[dst + w] = src[w];
    return;
  }
  const int64_t q = ((int64_t)blockIdx.x - a.G) * 256 + threadIdx.x;
  const int64_t n0 = a.count[a.b0];
  const int wd = 3 * a.b0 + 8;
  if (q >= (n0 * wd + 31) / 32 || 6 + q >= a.cap_words) return;
  const int64_t bit0 = 32 * q;
  const int64_t v_last = min(n0 - 1, (bit0 + 31) / wd);
  uint32_t word = 0;
  for (int64_t v = bit0 / wd; v <= v_last; ++v) {
    const uint64_t field = (uint64_t)(uint32_t)a.xyz[3 * v] | ((uint64_t)(uint32_t)a.xyz[3 * v + 1] << a.b0) |
                           ((uint64_t)(uint32_t)a.xyz[3 * v + 2] << (2 * a.b0)) |
                           ((uint64_t)a.code[v] << (3 * a.b0));
    const int64_t rel = v * wd - bit0;
    word |= rel >= 0 ? (uint32_t)(field << rel) : (uint32_t)(field >> (-rel));
  }
  a.out[6 + q] = word;
}

struct DecArgs {
  const uint32_t* words;  // the bitstream
  int64_t nwords;
  const int32_t* count;
  int b, L;
  const uint32_t* tab;  // [N_b][K] entries start | f << 16 of the scale's tables
  const uint8_t* s1;    // stage 2 of the two-stage head: S1 of every voxel (code = S1 | S2 << 4)
  uint8_t* out;         // [N_b] symbols (stage 2: the codes)
  uint64_t* fpos;       // [sections + 1] first word of each section
  int t;
  int64_t p0;  // first word of section 0
  int last;    // the frame's last section: its end must be the bitstream's
  uint32_t* err;
};

__device__ __forceinline__ int64_t wave_sum(int64_t v) {
  for (int d = 32; d >= 1; d >>= 1) {
    const int lo = __shfl_xor((int)(uint32_t)v, d), hi = __shfl_xor((int)(uint32_t)((uint64_t)v >> 32), d);
    v += (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
  }
  return v;
}


// The decoder's table of one voxel: entries start_s | f_s << 16 (start_0 =
// 0, ascending, f_s >= 1).  K = 256: four entries per lane (symbols 4l ..
// 4l + 3); K = 16: one entry in each of lanes 0 .. 15.
template <int K>
struct Table {
  uint32_t e[K == 256 ? 4 : 1];
};

template <int K>
__device__ __forceinline__ Table<K> load_table(const uint32_t* tab, int64_t i, int lane) {
  Table<K> r;
  if constexpr (K == 256) {
    const uint4 v = reinterpret_cast<const uint4*>(tab + i * 256)[lane];
    r.e[0] = v.x;
    r.e[1] = v.y;
    r.e[2] = v.z;
    r.e[3] = v.w;
  } else {
    r.e[0] = tab[i * 16 + (lane & 15)];
  }
  return r;
}

// The symbol s with start_s <= slot < start_s + f_s and its interval.  Every
// lane picks, among its own entries, the last one starting at or below slot
// (vector work that runs beside the scalar part), a ballot of "my first entry
// <= slot" names the lane holding s (starts ascend across the lanes), and
// two lane reads bring that lane's pick out.
template <int K>
__device__ __forceinline__ void find_symbol(const Table<K>& tb, uint32_t slot, uint32_t* sym, uint32_t* lo_s,
                                            uint32_t* f_s) {
  if constexpr (K == 256) {
    const bool c1 = (tb.e[1] & 0xFFFFu) <= slot, c2 = (tb.e[2] & 0xFFFFu) <= slot,
               c3 = (tb.e[3] & 0xFFFFu) <= slot;
    const uint32_t pick = c3 ? tb.e[3] : c2 ? tb.e[2] : c1 ? tb.e[1] : tb.e[0];
    const uint32_t k = c3 ? 3u : c2 ? 2u : c1 ? 1u : 0u;
    const uint64_t ball = __ballot((tb.e[0] & 0xFFFFu) <= slot);  // lane 0 always (its first entry is 0)
    const int ls = 63 - __clzll((long long)ball);
    const uint32_t a = rdl(pick, ls);
    *sym = 4u * (uint32_t)ls + rdl(k, ls);
    *lo_s = a & 0xFFFFu;
    *f_s = a >> 16;
  } else {
    const uint64_t ball = __ballot((tb.e[0] & 0xFFFFu) <= slot) & 0xFFFFull;
    const int ls = 63 - __clzll((long long)ball);
    const uint32_t a = rdl(tb.e[0], ls);
    *sym = (uint32_t)ls;
    *lo_s = a & 0xFFFFu;
    *f_s = a >> 16;
  }
}

// One wavefront per stream, in trips of 64 symbols.  A wavefront issues
// about one instruction per four cycles, so a stream's time is its symbol
// count times the instructions of one step: the step is kept short.  The
// coder state lives in scalar registers; a step reads its table from
// registers loaded kRing steps before (unconditional, clamped loads, so the
// compiler's wait names exactly that load), its renormalisation word from a
// register window of the stream (a lane read), and stores its symbol to LDS;
// the trip's symbols are written out together at its end (with the trip's S1
// values for stage 2).  Full trips run without per-step bounds; the last,
// partial trip checks them.  The window moves between trips only: a trip
// reads at most 64 words, from the two registers win0 and win1 (128 words),
// while the third, win2, is loaded a whole trip ahead (unconditionally, at
// a fixed point), so that no step waits on a window load issued after its
// own table loads.  A stream that runs past its end reads its last word
// again and is caught by the final check of its length and state.
template <int K, bool S1>
__global__ void __launch_bounds__(64 * kDecWaves) k_rans_decode(DecArgs a, const uint32_t* __restrict__ words,
                                                                const uint32_t* __restrict__ tab,
                                                                const uint8_t* __restrict__ s1,
                                                                uint8_t* __restrict__ out) {
  static_assert(64 % kRing == 0, "a trip holds whole turns of the table ring");
  __shared__ uint8_t s_sym[kDecWaves][64];
  const int lane = threadIdx.x & 63;
  // the wavefront index read through a lane read: the compiler then knows
  // that everything per stream is uniform and keeps it in scalar registers
  const int64_t wave = (int64_t)blockIdx.x * kDecWaves + (int64_t)rfl(threadIdx.x >> 6);
  const int64_t n = a.count[a.b];
  const int64_t S = streams_of(n, a.L);
  if (wave >= S) return;
  const int64_t start = a.t == 0 ? a.p0 : (int64_t)a.fpos[a.t];
  const int64_t hdr = (S + 1) / 2;
  if (start < 0 || start + hdr > a.nwords) {
    if (lane == 0) {
      latch(a.err, ERR_STREAM);
      if (wave == 0) a.fpos[a.t + 1] = (uint64_t)a.nwords + 1;  // later sections fail too
    }
    return;
  }
  // stream lengths: words before this stream (and, for stream 0, the section's total)
  auto len_of = [&](int64_t i) -> int64_t { return (words[start + i / 2] >> (16 * (i & 1))) & 0xFFFFu; };
  int64_t before = 0, all = 0;
  for (int64_t c0 = 0; c0 < (wave == 0 ? S : wave); c0 += 64) {
    const int64_t i = c0 + lane;
    const int64_t l = i < S ? len_of(i) : 0;
    before += i < wave ? l : 0;
    all += l;
  }
  before = wave_sum(before);
  if (wave == 0) {
    all = wave_sum(all);
    const int64_t end = start + hdr + all;
    if (lane == 0) {
      a.fpos[a.t + 1] = end <= a.nwords ? (uint64_t)end : (uint64_t)a.nwords + 1;
      if (end > a.nwords || (a.last && end != a.nwords)) latch(a.err, ERR_STREAM);
    }
  }
  const int64_t off = start + hdr + (int64_t)rfl((uint32_t)before) + ((int64_t)rfl((uint32_t)(before >> 32)) << 32);
  const int64_t len = (int64_t)rfl((uint32_t)len_of(wave));
  if (len < 2 || off + len > a.nwords) {
    if (lane == 0) latch(a.err, ERR_STREAM);
    return;
  }
  const uint32_t* in = words + off;
  // per-stream quantities in 32 bits (voxel indices stay below 2^31, a
  // stream below 2^16 words), so that their comparisons stay scalar
  const int ns = (int)n, Ss = (int)S, ws = (int)wave, lens = (int)len;
  const int m = ns > ws ? (ns - ws + Ss - 1) / Ss : 0;
  const int i_last = m > 0 ? ws + (m - 1) * Ss : 0;
  uint64_t x = ((uint64_t)in[0] << 32) | in[1];
  int p = 2;
  // renormalisation words: lane l of win0 holds word wb + l, win1 and win2
  // the next 64 each (the last word repeated past the stream's end, so that
  // the loads are unconditional)
  int wb = 2;
  auto word_at = [&](int q) -> uint32_t { return in[min(q, lens - 1)]; };
  uint32_t win0 = word_at(wb + lane), win1 = word_at(wb + 64 + lane);
  // both complete before any table load is issued: the trips' window reads
  // then never wait behind the table loads in flight
  __builtin_amdgcn_s_waitcnt(0);
  uint32_t win2 = word_at(wb + 128 + lane);
  Table<K> ring[kRing];
#pragma unroll
  for (int u = 0; u < kRing; ++u) ring[u] = load_table<K>(tab, min(ws + u * Ss, i_last), lane);
  int nidx = ws + kRing * Ss;  // the symbol whose table the next load fetches
  uint8_t* ssymb = s_sym[rfl(threadIdx.x >> 6)];
  // one trip; GUARD: the trip may hold fewer than 64 symbols (the last one)
  auto trip = [&](int k0, auto guard) {
    constexpr bool GUARD = decltype(guard)::value;
    const int i_mine = ws + (k0 + lane) * Ss;  // the symbol whose result lane `lane` writes
    const uint32_t s1v = S1 ? (uint32_t)s1[min(i_mine, i_last)] : 0u;
#pragma unroll
    for (int u = 0; u < 64; ++u) {
      // every step issues its load, so the count of loads in flight is the
      // same on every path and the wait for this step's table is exact
      const Table<K> cur = ring[u % kRing];
      ring[u % kRing] = load_table<K>(tab, min(nidx, i_last), lane);
      // advanced through a lane read, which the compiler cannot see through:
      // otherwise it keeps one address per unrolled step in scalar registers
      nidx = (int)rfl((uint32_t)(nidx + Ss));
      if (!GUARD || k0 + u < m) {
        const uint32_t slot = (uint32_t)x & ((1u << kProb) - 1u);
        uint32_t sym, lo_s, f_s;
        find_symbol<K>(cur, slot, &sym, &lo_s, &f_s);
        x = (uint64_t)f_s * (x >> kProb) + slot - lo_s;
        if ((uint32_t)(x >> 31) == 0) {  // x < 2^31 (x < 2^63 always)
          const int q = p - wb;          // below 128 inside a trip
          const uint32_t w0 = rdl(win0, q & 63), w1 = rdl(win1, q & 63);
          x = (x << 32) | (q < 64 ? w0 : w1);
          ++p;
        }
        // every lane stores the same byte: no lane mask to set up
        ssymb[u] = (uint8_t)sym;
      }
    }
    // LDS operations of one wavefront complete in order: the stores above
    // are visible here
    const uint32_t symv = ssymb[lane];
    if (!GUARD || k0 + lane < m) out[i_mine] = (uint8_t)(S1 ? (s1v | (symv << 4)) : symv);
    // the window moves on once its first 64 words are used up; win2 is
    // reloaded either way (the same words when the window did not move)
    const bool shift = p - wb >= 64;  // uniform
    win0 = shift ? win1 : win0;
    win1 = shift ? win2 : win1;
    wb = shift ? wb + 64 : wb;
    win2 = word_at(wb + 128 + lane);
  };
  const int full = m & ~63;
  for (int k0 = 0; k0 < full; k0 += 64) trip(k0, std::false_type{});
  if (full < m) trip(full, std::true_type{});
  if (lane == 0 && (p != lens || x != kLow)) latch(a.err, ERR_STREAM);
}

}  // namespace

int64_t rans_stream_bound(const Ctx& c, int sections, int L) {
  return (int64_t)sections * (c.cap_pts / L + 1);
}

hipError_t launch_rans_encode(Ctx& c, const uint16_t* iv, int b_lo, int b_hi, int stages, int L, uint32_t* region,
                              uint32_t* lens, int64_t G) {
  ProfScope ps_(c, RENO_K_ENTROPY);
  EncArgs a;
  a.iv = reinterpret_cast<const uint32_t*>(iv);
  a.count = c.d_count;
  a.moff = c.d_moff;
  a.cap_model = c.cap_model;
  a.b_lo = b_lo;
  a.sections = (b_hi - b_lo + 1) * stages;
  a.stages = stages;
  a.L = L;
  a.region = region;
  a.lens = lens;
  a.G = G;
  a.err = c.d_err;
  hipLaunchKernelGGL(k_rans_encode, dim3((unsigned)((G + kEncWaves - 1) / kEncWaves)), dim3(64 * kEncWaves), 0,
                     c.stream, a);
  return hipGetLastError();
}

hipError_t launch_rans_layout(Ctx& c, int b_lo, int b_hi, int stages, int L, int B, const uint32_t* lens,
                              int64_t G, int64_t* offs, uint32_t* out, int64_t cap_words, int64_t* total) {
  ProfScope ps_(c, RENO_K_ENTROPY);
  LayArgs a;
  a.count = c.d_count;
  a.b_lo = b_lo;
  a.sections = (b_hi - b_lo + 1) * stages;
  a.stages = stages;
  a.L = L;
  a.b0 = c.b0();
  a.B = B;
  a.lens = lens;
  a.G = G;
  a.offs = offs;
  a.out = out;
  a.cap_words = cap_words;
  a.total = total;
  a.err = c.d_err;
  hipLaunchKernelGGL(k_rans_layout, dim3(1), dim3(kLayThreads), 0, c.stream, a);
  return hipGetLastError();
}

hipError_t launch_rans_pack(Ctx& c, const uint32_t* region, const uint32_t* lens, const int64_t* offs, int L,
                            int64_t G, const int64_t* total, const int32_t* xyz, uint32_t* out, int64_t cap_words) {
  ProfScope ps_(c, RENO_K_ENTROPY);
  PackArgs a;
  a.region = region;
  a.lens = lens;
  a.offs = offs;
  a.total = total;
  a.L = L;
  a.G = G;
  a.xyz = xyz;
  a.code = c.lv_code + c.lv(c.b0());
  a.count = c.d_count;
  a.b0 = c.b0();
  a.out = out;
  a.cap_words = cap_words;
  const int64_t n0_max = std::min<int64_t>(c.cap_pts, int64_t(1) << (3 * c.b0()));
  const int64_t words_max = (n0_max * (3 * c.b0() + 8) + 31) / 32;
  hipLaunchKernelGGL(k_rans_pack, dim3((unsigned)(G + (words_max + 255) / 256)), dim3(256), 0, c.stream, a);
  return hipGetLastError();
}

hipError_t launch_rans_decode(Ctx& c, const uint32_t* words, int64_t nwords, int b, int L, int K,
                              const uint32_t* tab, const uint8_t* s1, uint8_t* out, uint64_t* fpos, int t,
                              int64_t p0, bool last) {
  ProfScope ps_(c, RENO_K_ENTROPY);
  DecArgs a;
  a.words = words;
  a.nwords = nwords;
  a.count = c.d_count;
  a.b = b;
  a.L = L;
  a.tab = tab;
  a.s1 = s1;
  a.out = out;
  a.fpos = fpos;
  a.t = t;
  a.p0 = p0;
  a.last = last ? 1 : 0;
  a.err = c.d_err;
  const int64_t waves = c.cap_pts / L + 1;
  const dim3 grid((unsigned)((waves + kDecWaves - 1) / kDecWaves));
  if (K == 256)
    hipLaunchKernelGGL((k_rans_decode<256, false>), grid, dim3(64 * kDecWaves), 0, c.stream, a, words, tab, s1,
                       out);
  else if (s1)
    hipLaunchKernelGGL((k_rans_decode<16, true>), grid, dim3(64 * kDecWaves), 0, c.stream, a, words, tab, s1, out);
  else
    hipLaunchKernelGGL((k_rans_decode<16, false>), grid, dim3(64 * kDecWaves), 0, c.stream, a, words, tab, s1,
                       out);
  return hipGetLastError();
}

}  // namespace reno
