// RENO hot-path oracle: a plain, slow, single-threaded CPU implementation of
// what the codec computes, written from the paper's definitions.
//
// TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the
// benchmark's CPU-baseline leg may load this library.  The GPU library shares
// no code, header, table or helper with it; both only consume the seeded
// inputs produced by the `synth` package.
//
// Representation: voxels are integer coordinate triples (x, y, z) kept in
// std::set / std::map; Morton keys are computed with a plain bit loop and are
// used for ordering only.  Floating point is double throughout, except where a
// step is defined on fp32 inputs (the points and the weights are fp32 data).
//
// Parity status of each function is stated next to it; every function here is
// pinned by a CPU test (see the test files named in the comments).
//
// Build: g++ -O2 -std=c++17 -ffp-contract=off -fPIC -shared oracle.cpp

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <set>
#include <vector>

namespace {

typedef std::array<int64_t, 3> Vox;

// Ordering of the voxels inside a scale.  The paper calls the codes
// "orderless" (Sec. 1) and fixes no order; the reading taken here is ascending
// bit-interleaved Morton order with x in the lowest bit of each triple
// (key = sum_i x_i 2^{3i} + y_i 2^{3i+1} + z_i 2^{3i+2}).  With it the children
// of a voxel v are 8 key(v) + delta, so the sorted next scale and the
// expansion order of the codes coincide.
uint64_t morton_loop(const Vox& v, int bits) {
  uint64_t k = 0;
  for (int i = 0; i < bits; ++i) {
    k |= (uint64_t)((v[0] >> i) & 1) << (3 * i);
    k |= (uint64_t)((v[1] >> i) & 1) << (3 * i + 1);
    k |= (uint64_t)((v[2] >> i) & 1) << (3 * i + 2);
  }
  return k;
}

struct ByKey {
  int bits;
  bool operator()(const Vox& a, const Vox& b) const {
    return morton_loop(a, bits) < morton_loop(b, bits);
  }
};

// One scale of the multiscale sparse tensor: the occupied coordinates C^d
// (Sec. 3, Eq. 1) and their occupancy codes O^d.
struct Level {
  int b = 0;                       // bit depth of this scale
  std::vector<Vox> v;              // voxels, ascending Morton order
  std::map<Vox, int64_t> row;      // voxel -> row in v
  std::vector<uint8_t> code;       // O_b (only for b < B)
  std::vector<int32_t> parent;     // row of v >> 1 in the scale below (-1 at b0)
};

struct Pyramid {
  int B = 0, b0 = 0;
  int64_t M = 0;                   // raw point count (0 when built from codes)
  std::vector<Level> lv;           // indexed by bit depth b (entries < b0 empty)
};

void finish_level(Level& L) {
  std::sort(L.v.begin(), L.v.end(), ByKey{L.b});
  L.row.clear();
  for (size_t i = 0; i < L.v.size(); ++i) L.row[L.v[i]] = (int64_t)i;
}

// Quantisation to the B-bit grid.  The paper states the precision only
// (+-8 mm at 14 bits, +-3.2 cm at 12 bits, Sec. 4.1.1 / Table 1).  Reading:
// the grid spans [-R, R) in 2^B cells of size 2R/2^B, floor binning,
// out-of-range values clamped to the edge cells; evaluated in fp64 exactly as
//   u = ((p + R) * 2^B) / (2R),   q = clamp(floor(u), 0, 2^B - 1).
// Non-finite input is an error.
int quantize_axis(float p, int B, double R, int64_t* q) {
  if (!std::isfinite(p)) return -1;
  double u = ((double)p + R) * (double)(int64_t(1) << B) / (2.0 * R);
  double f = std::floor(u);
  double top = (double)((int64_t(1) << B) - 1);
  if (f < 0.0) f = 0.0;
  if (f > top) f = top;
  *q = (int64_t)f;
  return 0;
}

// FOG (Sec. 3.1): the code of v is the sum over its eight children present in
// the finer scale of 2^delta, delta = dx + 2 dy + 4 dz.  Written as the
// membership test it stands for: a fixed-weight stride-2 convolution with
// weights 1, 2, ..., 128 over all-ones inputs.  The bit <-> octant assignment is
// the reading used throughout (the figure that would fix it is not available).
uint8_t fog_code(const Vox& v, const Level& finer) {
  unsigned code = 0;
  for (int d = 0; d < 8; ++d) {
    Vox c = {2 * v[0] + (d & 1), 2 * v[1] + ((d >> 1) & 1), 2 * v[2] + ((d >> 2) & 1)};
    if (finer.row.count(c)) code |= 1u << d;
  }
  return (uint8_t)code;
}

// Builds all scales b0..B from the finest voxel set (dyadic downscaling,
// Sec. 3: C^{d-1} = { floor(c / 2) : c in C^d }), the codes O_b for
// b0 <= b < B, and the parent rows.
void build_from_finest(Pyramid& P, const std::set<Vox>& finest) {
  P.lv.assign(P.B + 1, Level());
  for (int b = 0; b <= P.B; ++b) P.lv[b].b = b;
  P.lv[P.B].v.assign(finest.begin(), finest.end());
  finish_level(P.lv[P.B]);
  for (int b = P.B; b > P.b0; --b) {
    std::set<Vox> coarse;
    for (const Vox& v : P.lv[b].v) coarse.insert(Vox{v[0] >> 1, v[1] >> 1, v[2] >> 1});
    P.lv[b - 1].v.assign(coarse.begin(), coarse.end());
    finish_level(P.lv[b - 1]);
  }
  for (int b = P.b0; b < P.B; ++b) {
    Level& L = P.lv[b];
    L.code.resize(L.v.size());
    for (size_t i = 0; i < L.v.size(); ++i) L.code[i] = fog_code(L.v[i], P.lv[b + 1]);
  }
  for (int b = P.b0; b <= P.B; ++b) {
    Level& L = P.lv[b];
    L.parent.assign(L.v.size(), -1);
    if (b == P.b0) continue;
    for (size_t i = 0; i < L.v.size(); ++i) {
      Vox p = {L.v[i][0] >> 1, L.v[i][1] >> 1, L.v[i][2] >> 1};
      L.parent[i] = (int32_t)P.lv[b - 1].row.at(p);
    }
  }
}

// FCG (Sec. 3.1): expand each code into its eight bits and keep the children
// whose bit is 1.  Parents are visited in their stored order and, within a
// parent, children in ascending delta.
std::vector<Vox> fcg_expand(const std::vector<Vox>& v, const std::vector<uint8_t>& code) {
  std::vector<Vox> out;
  for (size_t i = 0; i < v.size(); ++i)
    for (int d = 0; d < 8; ++d)
      if ((code[i] >> d) & 1)
        out.push_back(Vox{2 * v[i][0] + (d & 1), 2 * v[i][1] + ((d >> 1) & 1),
                          2 * v[i][2] + ((d >> 2) & 1)});
  return out;
}

// Neighbour k of v at scale b for a ks x ks x ks kernel (ks odd, radius
// h = ks / 2): k = (dx+h) + ks(dy+h) + ks^2(dz+h), i.e. (dx+1) + 3(dy+1) +
// 9(dz+1) for ks = 3; the row of v + (dx,dy,dz) among the voxels of the
// scale, or -1 when that cell is empty or outside [0, 2^b)^3.
int64_t neighbour(const std::map<Vox, int64_t>& rows, int b, const Vox& v, int k, int ks = 3) {
  const int h = ks / 2;
  int dx = k % ks - h, dy = (k / ks) % ks - h, dz = k / (ks * ks) - h;
  Vox u = {v[0] + dx, v[1] + dy, v[2] + dz};
  int64_t lim = int64_t(1) << b;
  for (int a = 0; a < 3; ++a)
    if (u[a] < 0 || u[a] >= lim) return -1;
  auto it = rows.find(u);
  return it == rows.end() ? -1 : it->second;
}

// The ks^3 neighbour rows of voxel v (index k as above).
typedef std::vector<int64_t> Nbrs;
Nbrs neighbours_of(const std::map<Vox, int64_t>& rows, int b, const Vox& v, int ks = 3) {
  Nbrs nb(ks * ks * ks);
  for (int k = 0; k < ks * ks * ks; ++k) nb[k] = neighbour(rows, b, v, k, ks);
  return nb;
}

// One submanifold ks x ks x ks sparse convolution (stride 1, outputs only on
// the input voxels), as used by TOP's ResNet on the target coordinates (Eq. 9):
//   y(v)[co] = bias[co] + sum_k sum_ci W[k][ci][co] * h(nbr(v,k))[ci]
// over present neighbours, optionally followed by ReLU.  Cross-correlation
// convention, zero for absent neighbours.  `nb[r]` are the ks^3 neighbour rows
// of output r; `h` is indexed by row.
void sparse_conv(const std::vector<Nbrs>& nb, const std::vector<double>& h,
                 int c_in, const float* W, const float* bias, int c_out, bool relu,
                 std::vector<double>& y) {
  y.assign(nb.size() * c_out, 0.0);
  for (size_t r = 0; r < nb.size(); ++r) {
    const int kv = (int)nb[r].size();
    for (int co = 0; co < c_out; ++co) {
      double acc = (double)bias[co];
      for (int k = 0; k < kv; ++k) {
        int64_t n = nb[r][k];
        if (n < 0) continue;
        for (int ci = 0; ci < c_in; ++ci)
          acc += (double)W[((size_t)k * c_in + ci) * c_out + co] * h[n * c_in + ci];
      }
      y[r * c_out + co] = relu ? std::max(acc, 0.0) : acc;
    }
  }
}

}  // namespace

extern "C" {

struct OrcWeights {
  int c_in, channels, layers, pad;
  const float* conv_w[8];   // [27][C_in][C_out]
  const float* conv_b[8];   // [C_out]
  const float* head_w;      // [C][256]
  const float* head_b;      // [256]
  // bitwise two-stage head (Sec. 3.2, Eqs. 11-13), used when head_mode == 1
  int head_mode, pad2;
  const float* head1_w;     // [C][16]  stage 1 over S1 = O & 15
  const float* head1_b;     // [16]
  const float* emb_s1;      // [16][C]  Emb(S1), added to the features before stage 2
  const float* head2_w;     // [C][16]  stage 2 over S2 = O >> 4
  const float* head2_b;     // [16]
  // full target occupancy predictor (Sec. 3.2, Eqs. 6-9), used when model_mode == 1
  int model_mode, pad3;
  const float* emb_o;       // [256][C]  Emb(O^{d-1})
  const float* emb_d;       // [8][C]    Emb(delta)
  const float* top_w[4];    // [ks^3][C][C] residual blocks: A1, A2 (scale d-1), B1, B2 (scale d)
  const float* top_b[4];    // [C]
  int kernel_size, pad4;    // ks of the full predictor's convs (0 reads as 3)
};

uint64_t orc_morton(int64_t x, int64_t y, int64_t z, int bits) {
  return morton_loop(Vox{x, y, z}, bits);
}

// Quantises n points (fp32 xyz) to integer coordinates; returns -1 on a
// non-finite coordinate, else 0.
int orc_quantize(const float* pts, int64_t n, int B, double R, int64_t* q) {
  for (int64_t i = 0; i < 3 * n; ++i)
    if (quantize_axis(pts[i], B, R, &q[i]) != 0) return -1;
  return 0;
}

// Encoder side: quantise, deduplicate (the occupied coordinates, Sec. 3), build
// every scale down to b0 and the codes.  Returns NULL on bad input.
void* orc_pyramid_from_points(const float* pts, int64_t n, int B, int b0, double R) {
  if (B < 1 || B > 21 || b0 < 0 || b0 >= B) return nullptr;
  std::set<Vox> finest;
  for (int64_t i = 0; i < n; ++i) {
    Vox q;
    for (int a = 0; a < 3; ++a)
      if (quantize_axis(pts[3 * i + a], B, R, &q[a]) != 0) return nullptr;
    finest.insert(q);
  }
  Pyramid* P = new Pyramid();
  P->B = B;
  P->b0 = b0;
  P->M = n;
  build_from_finest(*P, finest);
  return P;
}

// Same, from integer voxels (duplicates allowed) of the finest scale.
void* orc_pyramid_from_voxels(const int64_t* xyz, int64_t n, int B, int b0) {
  if (B < 1 || B > 21 || b0 < 0 || b0 >= B) return nullptr;
  std::set<Vox> finest;
  int64_t lim = int64_t(1) << B;
  for (int64_t i = 0; i < n; ++i) {
    Vox q = {xyz[3 * i], xyz[3 * i + 1], xyz[3 * i + 2]};
    for (int a = 0; a < 3; ++a)
      if (q[a] < 0 || q[a] >= lim) return nullptr;
    finest.insert(q);
  }
  Pyramid* P = new Pyramid();
  P->B = B;
  P->b0 = b0;
  P->M = n;
  build_from_finest(*P, finest);
  return P;
}

// Decoder side (Eq. 2): start from the initial state (C^{b0}, O^{b0}) and apply
// FCG scale after scale with the codes O_{b0+1} .. O_{B-1}.  `codes` holds all
// of O_{b0} .. O_{B-1} concatenated in scale order; their count must match the
// expanded sizes, otherwise NULL is returned.
void* orc_pyramid_from_codes(const int64_t* base_xyz, int64_t n0, int b0, int B,
                             const uint8_t* codes, int64_t ncodes) {
  if (B < 1 || B > 21 || b0 < 0 || b0 >= B) return nullptr;
  Pyramid* P = new Pyramid();
  P->B = B;
  P->b0 = b0;
  P->lv.assign(B + 1, Level());
  for (int b = 0; b <= B; ++b) P->lv[b].b = b;
  for (int64_t i = 0; i < n0; ++i)
    P->lv[b0].v.push_back(Vox{base_xyz[3 * i], base_xyz[3 * i + 1], base_xyz[3 * i + 2]});
  int64_t used = 0;
  for (int b = b0; b < B; ++b) {
    Level& L = P->lv[b];
    if (b == b0) {
      L.row.clear();
      for (size_t i = 0; i < L.v.size(); ++i) L.row[L.v[i]] = (int64_t)i;
    }
    if (used + (int64_t)L.v.size() > ncodes) { delete P; return nullptr; }
    L.code.assign(codes + used, codes + used + L.v.size());
    used += (int64_t)L.v.size();
    Level& N = P->lv[b + 1];
    N.v = fcg_expand(L.v, L.code);
    N.row.clear();
    for (size_t i = 0; i < N.v.size(); ++i) N.row[N.v[i]] = (int64_t)i;
  }
  if (used != ncodes) { delete P; return nullptr; }
  for (int b = b0; b <= B; ++b) {
    Level& L = P->lv[b];
    L.parent.assign(L.v.size(), -1);
    if (b == b0) continue;
    for (size_t i = 0; i < L.v.size(); ++i) {
      Vox p = {L.v[i][0] >> 1, L.v[i][1] >> 1, L.v[i][2] >> 1};
      auto it = P->lv[b - 1].row.find(p);
      L.parent[i] = it == P->lv[b - 1].row.end() ? -1 : (int32_t)it->second;
    }
  }
  return P;
}

void orc_free(void* h) { delete static_cast<Pyramid*>(h); }

int64_t orc_num(void* h, int b) {
  Pyramid* P = static_cast<Pyramid*>(h);
  if (b < P->b0 || b > P->B) return -1;
  return (int64_t)P->lv[b].v.size();
}

int64_t orc_raw_points(void* h) { return static_cast<Pyramid*>(h)->M; }

void orc_xyz(void* h, int b, int64_t* out) {
  const Level& L = static_cast<Pyramid*>(h)->lv[b];
  for (size_t i = 0; i < L.v.size(); ++i)
    for (int a = 0; a < 3; ++a) out[3 * i + a] = L.v[i][a];
}

void orc_keys(void* h, int b, uint64_t* out) {
  const Level& L = static_cast<Pyramid*>(h)->lv[b];
  for (size_t i = 0; i < L.v.size(); ++i) out[i] = morton_loop(L.v[i], b);
}

// O_b for b0 <= b < B; returns -1 when the scale has no codes.
int orc_codes(void* h, int b, uint8_t* out) {
  Pyramid* P = static_cast<Pyramid*>(h);
  if (b < P->b0 || b >= P->B) return -1;
  const Level& L = P->lv[b];
  std::copy(L.code.begin(), L.code.end(), out);
  return 0;
}

void orc_parent(void* h, int b, int32_t* out) {
  const Level& L = static_cast<Pyramid*>(h)->lv[b];
  std::copy(L.parent.begin(), L.parent.end(), out);
}

// FCG applied to scale b of a pyramid with codes `codes` (N_b of them);
// writes the children as xyz triples and returns their count.
int64_t orc_expand(void* h, int b, const uint8_t* codes, int64_t* out_xyz) {
  const Level& L = static_cast<Pyramid*>(h)->lv[b];
  std::vector<uint8_t> c(codes, codes + L.v.size());
  std::vector<Vox> ch = fcg_expand(L.v, c);
  if (out_xyz)
    for (size_t i = 0; i < ch.size(); ++i)
      for (int a = 0; a < 3; ++a) out_xyz[3 * i + a] = ch[i][a];
  return (int64_t)ch.size();
}

// Neighbour map [N_b][ks^3] of scale b for kernel size ks (odd).
void orc_neighbors(void* h, int b, int ks, int32_t* out) {
  const Level& L = static_cast<Pyramid*>(h)->lv[b];
  const int kv = ks * ks * ks;
  for (size_t i = 0; i < L.v.size(); ++i)
    for (int k = 0; k < kv; ++k) out[i * kv + k] = (int32_t)neighbour(L.row, b, L.v[i], k, ks);
}

// Input features of the target voxels (target embedding, Eqs. 7-8, in the
// simplified form of the configured model): x_v = [delta bit 0, delta bit 1,
// delta bit 2, bits 0..7 of the parent's code], with delta = sum_k
// (c_k - 2 p_k) 2^{k-1} over x, y, z (the parent's coordinate taken in the
// child's frame).
void orc_features(void* h, int b, double* out /*[N][11]*/) {
  Pyramid* P = static_cast<Pyramid*>(h);
  const Level& L = P->lv[b];
  const Level& Pl = P->lv[b - 1];
  for (size_t i = 0; i < L.v.size(); ++i) {
    const Vox& c = L.v[i];
    const Vox& p = Pl.v[L.parent[i]];
    int delta = 0;
    for (int a = 0; a < 3; ++a) delta += (int)(c[a] - 2 * p[a]) << a;
    unsigned code = Pl.code[L.parent[i]];
    for (int j = 0; j < 3; ++j) out[i * 11 + j] = (double)((delta >> j) & 1);
    for (int j = 0; j < 8; ++j) out[i * 11 + 3 + j] = (double)((code >> j) & 1);
  }
}

// Standalone sparse conv on an explicit voxel list (rows in the given order),
// used to pin the layer against a dense 3D convolution.
int orc_sparse_conv(const int64_t* xyz, int64_t n, int bits, const double* feats, int c_in,
                    const float* W, const float* bias, int c_out, int relu, int ks, double* out) {
  if (ks < 1 || ks % 2 == 0) return -1;
  std::vector<Vox> v(n);
  std::map<Vox, int64_t> rows;
  for (int64_t i = 0; i < n; ++i) {
    v[i] = Vox{xyz[3 * i], xyz[3 * i + 1], xyz[3 * i + 2]};
    if (rows.count(v[i])) return -1;
    rows[v[i]] = i;
  }
  std::vector<double> h(feats, feats + n * c_in), y;
  std::vector<Nbrs> nb(n);
  for (int64_t i = 0; i < n; ++i) nb[i] = neighbours_of(rows, bits, v[i], ks);
  sparse_conv(nb, h, c_in, W, bias, c_out, relu != 0, y);
  std::copy(y.begin(), y.end(), out);
  return 0;
}

// TOP on scale b (Eq. 5 with the configured model): input features (above),
// L sparse conv + ReLU layers on the target coordinates, a linear head to 256
// logits (Eq. 10; 256 classes indexed by code value, class 0 kept in the
// normalisation although no code takes it), softmax, and the ideal code
// length -log2 p(O_b[v]) (Eq. 4).  Evaluated for the requested rows only:
// each layer is computed on the receptive field those rows need.
//   logits [nrows][256] (or NULL), lse [nrows] natural-log normaliser (or
//   NULL), bits [nrows] (or NULL; needs b < B).
// Residual block of the full predictor: x + conv2(ReLU(conv1(x))), then ReLU
// (3x3x3 submanifold convs C -> C with bias, on the neighbour lists nb).
static void res_block(const std::vector<Nbrs>& nb, const std::vector<double>& x, int C,
                      const float* w1, const float* b1, const float* w2, const float* b2,
                      std::vector<double>& out) {
  std::vector<double> t, y;
  sparse_conv(nb, x, C, w1, b1, C, true, t);
  sparse_conv(nb, t, C, w2, b2, C, false, y);
  out.resize(x.size());
  for (size_t i = 0; i < x.size(); ++i) out[i] = std::max(x[i] + y[i], 0.0);
}

// Full target occupancy predictor (Sec. 3.2), in this reading of Eqs. 6-9:
//   F^{d-1} = RB_A(C^{d-1}, Emb_O[O^{d-1}])                 occupancy features (Eq. 6)
//   X^d(v)  = F^{d-1}(parent(v)) + Emb_D[delta(v)]           replication + octant (Eqs. 7-9)
//   F^d     = RB_B(C^d, X^d)                                  (Eq. 9)
// evaluated on every voxel of scales b-1 and b; cur = F^b [N_b][C].
static int top_features(Pyramid* P, int b, const OrcWeights* w, std::vector<double>& cur) {
  const Level& L = P->lv[b];
  const Level& Pl = P->lv[b - 1];
  const int C = w->channels;
  const int64_t Np = (int64_t)Pl.v.size(), N = (int64_t)L.v.size();
  const int ks = w->kernel_size > 0 ? w->kernel_size : 3;
  std::vector<Nbrs> nbA(Np), nbB(N);
  for (int64_t u = 0; u < Np; ++u) nbA[u] = neighbours_of(Pl.row, b - 1, Pl.v[u], ks);
  for (int64_t v = 0; v < N; ++v) nbB[v] = neighbours_of(L.row, b, L.v[v], ks);
  std::vector<double> xa(Np * C), fa, xb(N * C);
  for (int64_t u = 0; u < Np; ++u)
    for (int c = 0; c < C; ++c) xa[u * C + c] = (double)w->emb_o[(size_t)Pl.code[u] * C + c];
  res_block(nbA, xa, C, w->top_w[0], w->top_b[0], w->top_w[1], w->top_b[1], fa);
  for (int64_t v = 0; v < N; ++v) {
    const Vox& c0 = L.v[v];
    const int64_t p = L.parent[v];
    const Vox& pv = Pl.v[p];
    int delta = 0;
    for (int a = 0; a < 3; ++a) delta += (int)(c0[a] - 2 * pv[a]) << a;
    for (int c = 0; c < C; ++c) xb[v * C + c] = fa[p * C + c] + (double)w->emb_d[delta * C + c];
  }
  res_block(nbB, xb, C, w->top_w[2], w->top_b[2], w->top_w[3], w->top_b[3], cur);
  return 0;
}

// Features h_L of the last conv layer for the requested rows, stored densely
// over all N rows of the scale in `cur` ([N][C]; rows outside the requested
// set are zero, except for the full predictor, which evaluates every row).
// Returns -1 on bad arguments.
static int final_features(void* h, int b, const OrcWeights* w, const int64_t* rows, int64_t nrows,
                   std::vector<double>& cur) {
  Pyramid* P = static_cast<Pyramid*>(h);
  if (b <= P->b0 || b > P->B) return -1;
  if (w->model_mode == 1) {
    for (int64_t i = 0; i < nrows; ++i)
      if (rows[i] < 0 || rows[i] >= (int64_t)P->lv[b].v.size()) return -1;
    return top_features(P, b, w, cur);
  }
  if (w->layers < 1 || w->layers > 8) return -1;
  const Level& L = P->lv[b];
  const int C = w->channels;
  const int64_t N = (int64_t)L.v.size();
  // receptive fields: need[l] = rows whose layer-l output is required
  std::vector<std::vector<int64_t>> need(w->layers + 1);
  std::vector<char> mark(N, 0);
  for (int64_t i = 0; i < nrows; ++i) {
    if (rows[i] < 0 || rows[i] >= N) return -1;
    if (!mark[rows[i]]) { mark[rows[i]] = 1; need[w->layers].push_back(rows[i]); }
  }
  std::map<int64_t, Nbrs> nbmap;   // neighbour rows, computed once per row
  auto nbrs = [&](int64_t r) -> const Nbrs& {
    auto it = nbmap.find(r);
    if (it == nbmap.end()) it = nbmap.emplace(r, neighbours_of(L.row, b, L.v[r])).first;
    return it->second;
  };
  for (int l = w->layers; l > 0; --l) {
    std::fill(mark.begin(), mark.end(), 0);
    for (int64_t r : need[l])
      for (int k = 0; k < 27; ++k) {
        int64_t nb = nbrs(r)[k];
        if (nb >= 0 && !mark[nb]) { mark[nb] = 1; need[l - 1].push_back(nb); }
      }
    std::sort(need[l - 1].begin(), need[l - 1].end());
  }
  // layer-0 features on need[0]; activations are stored densely over all N
  // rows (zeros elsewhere, never read)
  std::vector<double> x(N * 11, 0.0), feat_all(N * 11);
  orc_features(h, b, feat_all.data());
  for (int64_t r : need[0])
    for (int j = 0; j < 11; ++j) x[r * 11 + j] = feat_all[r * 11 + j];
  cur = x;
  std::vector<double> y;
  int c_in = 11;
  for (int l = 1; l <= w->layers; ++l) {
    std::vector<int64_t> out_rows = need[l];
    std::sort(out_rows.begin(), out_rows.end());
    std::vector<Nbrs> nb;
    for (int64_t r : out_rows) nb.push_back(nbrs(r));
    sparse_conv(nb, cur, c_in, w->conv_w[l - 1], w->conv_b[l - 1], C, true, y);
    std::vector<double> nxt(N * C, 0.0);
    for (size_t r = 0; r < out_rows.size(); ++r)
      for (int c = 0; c < C; ++c) nxt[out_rows[r] * C + c] = y[r * C + c];
    cur.swap(nxt);
    c_in = C;
  }
  return 0;
}

// Natural-log normaliser of a logit vector (max subtracted first).
static double log_sum_exp(const double* z, int n) {
  double m = z[0];
  for (int s = 1; s < n; ++s) m = std::max(m, z[s]);
  double sum = 0.0;
  for (int s = 0; s < n; ++s) sum += std::exp(z[s] - m);
  return m + std::log(sum);
}

int orc_model(void* h, int b, const OrcWeights* w, const int64_t* rows, int64_t nrows,
              double* logits, double* lse, double* bits) {
  Pyramid* P = static_cast<Pyramid*>(h);
  if (bits && b >= P->B) return -1;
  std::vector<double> cur;
  if (final_features(h, b, w, rows, nrows, cur) != 0) return -1;
  const Level& L = P->lv[b];
  const int C = w->channels;
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t r = rows[i];
    double z[256];
    for (int s = 0; s < 256; ++s) {
      double acc = (double)w->head_b[s];
      for (int c = 0; c < C; ++c) acc += (double)w->head_w[c * 256 + s] * cur[r * C + c];
      z[s] = acc;
    }
    const double l = log_sum_exp(z, 256);
    if (logits) for (int s = 0; s < 256; ++s) logits[i * 256 + s] = z[s];
    if (lse) lse[i] = l;
    if (bits) bits[i] = (l - z[L.code[r]]) / std::log(2.0);
  }
  return 0;
}

// Bitwise two-stage head (Sec. 3.2, Eqs. 11-13; linear MLPs in this model):
// the code O splits into S1 = O & 15 (children delta = 0..3, coded first) and
// S2 = O >> 4 (delta = 4..7), and P(O) = P(S1) P(S2 | S1) with
//   z1 = head1_w^T h + head1_b,                 P(S1)      = softmax(z1)
//   z2 = head2_w^T (h + emb_s1[S1]) + head2_b,  P(S2 | S1) = softmax(z2).
// S1 is taken from `s1` ([nrows], values 0..15) when given, else from O_b.
//   logits1 / logits2 [nrows][16], lse1 / lse2 [nrows] (each may be NULL),
//   bits [nrows] = -log2 P(S1) - log2 P(S2 | S1) (or NULL; needs b < B and
//   S1 from O_b).
int orc_model2(void* h, int b, const OrcWeights* w, const int64_t* rows, int64_t nrows,
               const uint8_t* s1, double* logits1, double* logits2, double* lse1, double* lse2,
               double* bits) {
  Pyramid* P = static_cast<Pyramid*>(h);
  if (w->head_mode != 1) return -1;
  if ((bits || !s1) && b >= P->B) return -1;
  if (bits && s1) return -1;
  std::vector<double> cur;
  if (final_features(h, b, w, rows, nrows, cur) != 0) return -1;
  const Level& L = P->lv[b];
  const int C = w->channels;
  for (int64_t i = 0; i < nrows; ++i) {
    const int64_t r = rows[i];
    const int a = s1 ? s1[i] : (L.code[r] & 15);
    if (a < 0 || a > 15) return -1;
    double z1[16], z2[16];
    for (int s = 0; s < 16; ++s) {
      double acc = (double)w->head1_b[s];
      for (int c = 0; c < C; ++c) acc += (double)w->head1_w[c * 16 + s] * cur[r * C + c];
      z1[s] = acc;
    }
    for (int s = 0; s < 16; ++s) {
      double acc = (double)w->head2_b[s];
      for (int c = 0; c < C; ++c)
        acc += (double)w->head2_w[c * 16 + s] * (cur[r * C + c] + (double)w->emb_s1[a * C + c]);
      z2[s] = acc;
    }
    const double l1 = log_sum_exp(z1, 16), l2 = log_sum_exp(z2, 16);
    if (logits1) for (int s = 0; s < 16; ++s) logits1[i * 16 + s] = z1[s];
    if (logits2) for (int s = 0; s < 16; ++s) logits2[i * 16 + s] = z2[s];
    if (lse1) lse1[i] = l1;
    if (lse2) lse2[i] = l2;
    if (bits) bits[i] = ((l1 - z1[a]) + (l2 - z2[L.code[r] >> 4])) / std::log(2.0);
  }
  return 0;
}

// Code-length totals (Eqs. 3-4): per_scale[b] = sum over V_b of the ideal bits
// for b0 < b < B; per_scale[b0] = the raw cost of the initial state
// (32-bit count + 3*b0 bits per coordinate + 8 bits per code, a reading: the
// paper leaves the coding of (C^0, O^0) open).  Returns the total T.
double orc_totals(void* h, const OrcWeights* w, double* per_scale /*[B+1] or NULL*/) {
  Pyramid* P = static_cast<Pyramid*>(h);
  double T = 32.0 + (double)P->lv[P->b0].v.size() * (3.0 * P->b0 + 8.0);
  if (per_scale) {
    for (int b = 0; b <= P->B; ++b) per_scale[b] = 0.0;
    per_scale[P->b0] = T;
  }
  for (int b = P->b0 + 1; b < P->B; ++b) {
    const int64_t N = (int64_t)P->lv[b].v.size();
    std::vector<int64_t> rows(N);
    for (int64_t i = 0; i < N; ++i) rows[i] = i;
    std::vector<double> bits(N);
    const int rc = w->head_mode == 1
                       ? orc_model2(h, b, w, rows.data(), N, nullptr, nullptr, nullptr, nullptr,
                                    nullptr, bits.data())
                       : orc_model(h, b, w, rows.data(), N, nullptr, nullptr, bits.data());
    if (rc != 0) return -1.0;
    double s = 0.0;
    for (double v : bits) s += v;
    if (per_scale) per_scale[b] = s;
    T += s;
  }
  return T;
}

// ---------------------------------------------------------------------------
// rANS (Duda, "Asymmetric numeral systems", arXiv:1311.2540), used to check
// that the ideal code lengths are achievable and that coding is lossless.
// State x in [2^31, 2^63), 32-bit renormalisation words, 16-bit probability
// precision: a symbol with start s and frequency f (sum of f <= 2^16) maps
//   x -> floor(x / f) * 2^16 + (x mod f) + s.
// Symbols are encoded in reverse so that the decoder emits them forward.
// Frequencies from probabilities over K symbols: f = 1 + floor(p * (2^16 - 2K))
// in fp32 (65024 for K = 256, 65504 for the 16-way stages of the two-stage
// head), and the 2^16 - sum(f) leftover slots go to the lowest-index most
// frequent symbol.

void orc_freqs_from_probs_k(const double* p, int k, uint32_t* f) {
  const float scale = (float)(65536 - 2 * k);
  uint32_t sum = 0;
  for (int s = 0; s < k; ++s) {
    float pf = (float)p[s];
    f[s] = 1u + (uint32_t)std::floor(pf * scale);
    sum += f[s];
  }
  int best = 0;
  for (int s = 1; s < k; ++s)
    if (f[s] > f[best]) best = s;
  f[best] += 65536u - sum;
}

void orc_freqs_from_probs(const double* p, uint32_t* f) { orc_freqs_from_probs_k(p, 256, f); }

// Encodes n symbols; freq [n][256]; writes 32-bit words to out (capacity
// `cap`), returns the number of words or -1.
int64_t orc_rans_encode(const uint8_t* sym, const uint32_t* freq, int64_t n, uint32_t* out,
                        int64_t cap) {
  std::vector<uint32_t> words;
  uint64_t x = uint64_t(1) << 31;
  for (int64_t i = n - 1; i >= 0; --i) {
    const uint32_t* f = freq + i * 256;
    uint64_t start = 0;
    for (int s = 0; s < sym[i]; ++s) start += f[s];
    uint64_t fs = f[sym[i]];
    if (fs == 0) return -1;
    // keep floor(x / fs) * 2^16 below 2^63
    uint64_t x_max = (uint64_t(1) << 47) * fs;
    while (x >= x_max) { words.push_back((uint32_t)x); x >>= 32; }
    x = (x / fs) * 65536u + (x % fs) + start;
  }
  words.push_back((uint32_t)x);
  words.push_back((uint32_t)(x >> 32));
  if ((int64_t)words.size() > cap) return -1;
  // stream is read back to front by the decoder
  for (size_t i = 0; i < words.size(); ++i) out[i] = words[words.size() - 1 - i];
  return (int64_t)words.size();
}

int orc_rans_decode(const uint32_t* in, int64_t nwords, const uint32_t* freq, int64_t n,
                    uint8_t* sym) {
  if (nwords < 2) return -1;
  int64_t pos = 0;
  uint64_t x = ((uint64_t)in[0] << 32) | in[1];
  pos = 2;
  for (int64_t i = 0; i < n; ++i) {
    const uint32_t* f = freq + i * 256;
    uint32_t slot = (uint32_t)(x & 0xFFFF);
    uint32_t start = 0;
    int s = 0;
    while (s < 255 && start + f[s] <= slot) { start += f[s]; ++s; }
    if (slot < start || slot >= start + f[s]) return -1;
    sym[i] = (uint8_t)s;
    x = (uint64_t)f[s] * (x >> 16) + slot - start;
    while (x < (uint64_t(1) << 31)) {
      if (pos >= nwords) return -1;
      x = (x << 32) | in[pos++];
    }
  }
  return pos == nwords ? 0 : -1;
}

}  // extern "C"
