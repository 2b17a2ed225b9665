// ocref: plain CPU oracle of the O-CNN octree hot path.
//
// TEST INFRASTRUCTURE ONLY.  Nothing in the product path links, loads or
// calls this file; it exists so that tests, the package smoke check and the
// bench's CPU-baseline leg can check the HIP library against an independent,
// slow, obviously correct implementation written from the paper
// (Wang et al., "O-CNN", arXiv 1712.01537).  It shares no source, header,
// table or helper with the HIP library.
//
// Every function follows the paper's literal statement of the step:
//   * octree: breadth-first subdivision of non-empty octants (Sec. 3.1,
//     "Octree construction"), shuffle keys (Sec. 3.1, "Shuffle key"), labels
//     (Sec. 3.1, "Label"), super-octree keys/labels (Sec. 3.1, "Mini-batch");
//   * input signal: mean normal per non-empty leaf (Sec. 3.1, "Input signal");
//   * neighbours: per-octant hash lookup of the K^3 neighbour keys
//     (Sec. 3.2, "3D Convolution", hash table H: key -> index);
//   * convolution: unrolled form (Sec. 3.2 equation for Phi_c) as im2col
//     followed by a matrix product, absent neighbours read as zero; backward as
//     the transposed products with a col2im scatter-add;
//   * stride-2 convolution on the first sibling, renewed through L_{l-1}
//     (Sec. 3.2, stride paragraphs; Fig. 2(d));
//   * max-pooling over 8 contiguous siblings, scattered through L_{l-1},
//     switches kept for unpooling (Sec. 3.2 "Pooling", "Unpooling", Fig. 5).
// All accumulation is in double.
//
// Parity pins (tests/test_oracle_*.py): hand-checked keys, the Fig. 2
// worked example in 3D, brute-force occupancy and neighbour matches, dense
// torch conv3d / max_pool3d / max_unpool3d in float64, autograd, finite
// differences and the adjoint identity.

#include <omp.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <unordered_map>
#include <unordered_set>
#include <vector>

namespace {

enum { OK = 0, ERR_ARG = 1, ERR_RANGE = 2 };

// Sec. 3.1 "Shuffle key": key(O) = x1 y1 z1 x2 y2 z2 ... xl yl zl, where
// x1 is the most significant bit of x (so child index c = 4x + 2y + z).
uint32_t shuffle_key(uint32_t x, uint32_t y, uint32_t z, int l) {
  uint32_t key = 0;
  for (int i = 1; i <= l; ++i) {
    int bit = l - i;  // x_i is bit (l - i) of x
    uint32_t xi = (x >> bit) & 1u, yi = (y >> bit) & 1u, zi = (z >> bit) & 1u;
    key = (key << 3) | (xi << 2) | (yi << 1) | zi;
  }
  return key;
}

// Inverse of shuffle_key: read the l triples from the top.
void key_coords(uint32_t key, int l, int64_t* x, int64_t* y, int64_t* z) {
  int64_t X = 0, Y = 0, Z = 0;
  for (int i = 1; i <= l; ++i) {
    uint32_t g = (key >> (3 * (l - i))) & 7u;
    X = (X << 1) | ((g >> 2) & 1u);
    Y = (Y << 1) | ((g >> 1) & 1u);
    Z = (Z << 1) | (g & 1u);
  }
  *x = X;
  *y = Y;
  *z = Z;
}

// Super-octree key (Sec. 3.1 "Mini-batch"): object index in the top 8 bits.
uint32_t super_key(uint32_t b, uint32_t key) { return (b << 24) | key; }

struct Level {
  std::vector<uint32_t> key;   // super keys, ascending
  std::vector<int32_t> label;  // 0 = empty, p = p-th non-empty octant (1-based)
  std::vector<int32_t> rows;   // rows[p-1] = index of the octant with label p
};

struct Tree {
  int depth = 0, full_depth = 0, batch = 0;
  std::vector<Level> lv;
  std::vector<float> signal;  // [N_d][3]
};

}  // namespace

extern "C" {

// Build the super-octree of B shapes.  points/normals: host f32 [P][3];
// offsets: host i32 [B+1], shape b owns points offsets[b]..offsets[b+1]-1.
int ocref_build(const float* points, const float* normals, const int32_t* offsets, int32_t batch,
                int32_t depth, int32_t full_depth, void** out) {
  if (!out) return ERR_ARG;
  *out = nullptr;
  if (batch < 1 || batch > 256 || depth < 1 || depth > 8 || full_depth < 0 || full_depth > depth ||
      !offsets)
    return ERR_ARG;
  if (offsets[0] != 0) return ERR_ARG;
  for (int b = 0; b < batch; ++b)
    if (offsets[b + 1] < offsets[b]) return ERR_ARG;
  const int64_t P = offsets[batch];
  if (P > 0 && (!points || !normals)) return ERR_ARG;

  // Quantise each point at the leaf depth: q = min(floor(p * 2^d), 2^d - 1),
  // evaluated in fp32 (scaling by a power of two is exact).
  const float scale = std::ldexp(1.0f, depth);
  const uint32_t qmax = (1u << depth) - 1u;
  std::vector<uint32_t> q(3 * P);
  for (int64_t i = 0; i < 3 * P; ++i) {
    float p = points[i];
    if (!(p >= 0.0f && p <= 1.0f)) return ERR_RANGE;  // also rejects NaN
    float v = p * scale;
    uint32_t c = (uint32_t)std::floor(v);
    q[i] = c > qmax ? qmax : c;
  }
  // Normals are averaged into the input signal: they must be finite.
  for (int64_t i = 0; i < 3 * P; ++i)
    if (!std::isfinite(normals[i])) return ERR_RANGE;
  std::vector<int32_t> shape_of(P);
  for (int b = 0; b < batch; ++b)
    for (int64_t i = offsets[b]; i < offsets[b + 1]; ++i) shape_of[i] = b;

  // occupied[l]: super keys of the depth-l octants that contain a point.
  std::vector<std::unordered_set<uint32_t>> occupied(depth + 1);
  for (int64_t i = 0; i < P; ++i)
    for (int l = 0; l <= depth; ++l) {
      int sh = depth - l;
      occupied[l].insert(super_key(shape_of[i], shuffle_key(q[3 * i] >> sh, q[3 * i + 1] >> sh,
                                                            q[3 * i + 2] >> sh, l)));
    }

  Tree* t = new Tree;
  t->depth = depth;
  t->full_depth = full_depth;
  t->batch = batch;
  t->lv.resize(depth + 1);

  // Depth 0: one root per shape.  Depths below full_depth are forced
  // non-empty (Sec. 4: all octants of the 2nd depth exist).
  {
    Level& L0 = t->lv[0];
    int32_t next = 0;
    for (int b = 0; b < batch; ++b) {
      uint32_t k = super_key(b, 0);
      bool nonempty = occupied[0].count(k) > 0 || 0 < full_depth;
      L0.key.push_back(k);
      L0.label.push_back(nonempty ? ++next : 0);
      if (nonempty) L0.rows.push_back(b);
    }
  }
  // Breadth-first subdivision: every non-empty octant at depth l gets its 8
  // children at depth l+1, in key order; labels are a running count over the
  // whole super-octree.
  for (int l = 0; l < depth; ++l) {
    const Level& P_ = t->lv[l];
    Level& C = t->lv[l + 1];
    int32_t next = 0;
    for (size_t j = 0; j < P_.key.size(); ++j) {
      if (P_.label[j] == 0) continue;
      uint32_t b = P_.key[j] >> 24, k = P_.key[j] & 0xFFFFFFu;
      for (uint32_t c = 0; c < 8; ++c) {
        uint32_t ck = super_key(b, k * 8u + c);
        bool nonempty = occupied[l + 1].count(ck) > 0 || (l + 1) < full_depth;
        C.label.push_back(nonempty ? ++next : 0);
        if (nonempty) C.rows.push_back((int32_t)C.key.size());
        C.key.push_back(ck);
      }
    }
  }

  // Input signal (Sec. 3.1): mean normal of the points in each non-empty
  // leaf, zero for empty leaves.
  const Level& Ld = t->lv[depth];
  std::unordered_map<uint32_t, int64_t> leaf_row;
  for (size_t i = 0; i < Ld.key.size(); ++i) leaf_row[Ld.key[i]] = (int64_t)i;
  std::vector<double> sum(3 * Ld.key.size(), 0.0);
  std::vector<int64_t> cnt(Ld.key.size(), 0);
  for (int64_t i = 0; i < P; ++i) {
    uint32_t k = super_key(shape_of[i], shuffle_key(q[3 * i], q[3 * i + 1], q[3 * i + 2], depth));
    int64_t r = leaf_row.at(k);
    for (int a = 0; a < 3; ++a) sum[3 * r + a] += (double)normals[3 * i + a];
    cnt[r] += 1;
  }
  t->signal.assign(3 * Ld.key.size(), 0.0f);
  for (size_t r = 0; r < Ld.key.size(); ++r)
    if (cnt[r] > 0)
      for (int a = 0; a < 3; ++a) t->signal[3 * r + a] = (float)(sum[3 * r + a] / (double)cnt[r]);

  *out = t;
  return OK;
}

void ocref_free(void* t) { delete static_cast<Tree*>(t); }

int ocref_level_size(const void* tp, int32_t l, int64_t* n, int64_t* m) {
  const Tree* t = static_cast<const Tree*>(tp);
  if (!t || l < 0 || l > t->depth) return ERR_ARG;
  *n = (int64_t)t->lv[l].key.size();
  *m = (int64_t)t->lv[l].rows.size();
  return OK;
}

// Copy S_l (super keys), L_l (labels) and the label -> row map of depth l.
int ocref_level(const void* tp, int32_t l, uint32_t* keys, int32_t* labels, int32_t* rows) {
  const Tree* t = static_cast<const Tree*>(tp);
  if (!t || l < 0 || l > t->depth) return ERR_ARG;
  const Level& L = t->lv[l];
  if (keys) std::memcpy(keys, L.key.data(), L.key.size() * sizeof(uint32_t));
  if (labels) std::memcpy(labels, L.label.data(), L.label.size() * sizeof(int32_t));
  if (rows) std::memcpy(rows, L.rows.data(), L.rows.size() * sizeof(int32_t));
  return OK;
}

int ocref_signal(const void* tp, float* sig) {
  const Tree* t = static_cast<const Tree*>(tp);
  if (!t || !sig) return ERR_ARG;
  std::memcpy(sig, t->signal.data(), t->signal.size() * sizeof(float));
  return OK;
}

// Neighbour search (Sec. 3.2): restore (x,y,z) from the key, offset it,
// re-encode, look the key up in H: key -> index over all octants of depth l.
// Offset index k = ((dx+r)*K + (dy+r))*K + (dz+r), r = (K-1)/2.
// stride 1: one row per octant of depth l, nb [N_l][K^3].
// stride 2^r (r >= 1): one row per non-empty octant p of depth l-r, in label
//           order, centred on the first depth-l octant of the sub-tree of
//           height r below p (Sec. 3.2, stride paragraphs): position
//           2^r * (coordinates of p), whether or not an octant is stored
//           there; nb [M_{l-r}][K^3].  For r = 1 that is p's first child.
// Missing neighbours (outside the cube, or not in the octree) are -1.
int ocref_neighbors(const void* tp, int32_t l, int32_t K, int32_t stride, int32_t* nb) {
  const Tree* t = static_cast<const Tree*>(tp);
  if (!t || !nb || l < 0 || l > t->depth || K < 1 || (K % 2) == 0 || stride < 1 ||
      (stride & (stride - 1)) != 0)
    return ERR_ARG;
  int sr = 0;
  while ((1 << sr) < stride) ++sr;
  if (sr > l) return ERR_ARG;
  const Level& L = t->lv[l];
  std::unordered_map<uint32_t, int32_t> H;
  H.reserve(L.key.size() * 2);
  for (size_t i = 0; i < L.key.size(); ++i) H[L.key[i]] = (int32_t)i;

  const int r = (K - 1) / 2, K3 = K * K * K;
  const int64_t side = int64_t(1) << l;
  const int64_t n_out = stride == 1 ? (int64_t)L.key.size() : (int64_t)t->lv[l - sr].rows.size();
#pragma omp parallel for schedule(static)
  for (int64_t o = 0; o < n_out; ++o) {
    uint32_t b;
    int64_t x, y, z;
    if (stride == 1) {
      b = L.key[o] >> 24;
      key_coords(L.key[o] & 0xFFFFFFu, l, &x, &y, &z);
    } else {  // the o-th non-empty octant of depth l - sr, scaled to depth l
      const Level& P = t->lv[l - sr];
      const uint32_t key = P.key[P.rows[o]];
      b = key >> 24;
      key_coords(key & 0xFFFFFFu, l - sr, &x, &y, &z);
      x <<= sr, y <<= sr, z <<= sr;
    }
    for (int dx = -r; dx <= r; ++dx)
      for (int dy = -r; dy <= r; ++dy)
        for (int dz = -r; dz <= r; ++dz) {
          int k = ((dx + r) * K + (dy + r)) * K + (dz + r);
          int64_t X = x + dx, Y = y + dy, Z = z + dz;
          int32_t row = -1;
          if (X >= 0 && X < side && Y >= 0 && Y < side && Z >= 0 && Z < side) {
            auto it = H.find(super_key(b, shuffle_key((uint32_t)X, (uint32_t)Y, (uint32_t)Z, l)));
            if (it != H.end()) row = it->second;
          }
          nb[o * K3 + k] = row;
        }
  }
  return OK;
}

// Convolution forward (Sec. 3.2, unrolled form): im2col row
// col[i][k*cin+ci] = X[nb[i][k]][ci] (0 when absent), then Y[i] = col[i] . W,
// W laid out [K^3][cin][cout].  rows (nullable): compute only these output
// rows, y is then [nrows][cout]; otherwise y is [n_out][cout].
int ocref_conv_fwd(const int32_t* nb, int64_t n_out, int32_t K3, const double* x, int64_t n_in,
                   int32_t cin, const double* w, int32_t cout, const int64_t* rows, int64_t nrows,
                   double* y) {
  if (!nb || !x || !w || !y || K3 < 1 || cin < 1 || cout < 1) return ERR_ARG;
  const int64_t n = rows ? nrows : n_out;
  for (int64_t o = 0; o < n; ++o)
    if (rows && (rows[o] < 0 || rows[o] >= n_out)) return ERR_ARG;
#pragma omp parallel
  {
    std::vector<double> col((size_t)K3 * cin);
#pragma omp for schedule(static)
    for (int64_t o = 0; o < n; ++o) {
      const int64_t i = rows ? rows[o] : o;
      for (int k = 0; k < K3; ++k) {
        int32_t j = nb[i * K3 + k];
        for (int ci = 0; ci < cin; ++ci)
          col[(size_t)k * cin + ci] = (j >= 0 && j < n_in) ? x[j * cin + ci] : 0.0;
      }
      for (int co = 0; co < cout; ++co) {
        double acc = 0.0;
        for (int64_t kc = 0; kc < (int64_t)K3 * cin; ++kc) acc += col[kc] * w[kc * cout + co];
        y[o * cout + co] = acc;
      }
    }
  }
  return OK;
}

// Convolution backward w.r.t. the input: dcol[i] = dY[i] . W^T, then col2im,
// a serial scatter-add of dcol[i][k] into row nb[i][k] in (i, k) order.
// Threads split the input channels (a channel's entries see the same
// additions in the same order at any thread count).  want (nullable,
// [n_in]): only accumulate into rows with want[j] != 0 (others stay 0).
int ocref_conv_bwd_data(const int32_t* nb, int64_t n_out, int32_t K3, const double* dy,
                        int32_t cout, const double* w, int32_t cin, int64_t n_in,
                        const uint8_t* want, double* dx) {
  if (!nb || !dy || !w || !dx || K3 < 1 || cin < 1 || cout < 1) return ERR_ARG;
  std::fill(dx, dx + n_in * cin, 0.0);
#pragma omp parallel
  {
    const int64_t nt = omp_get_num_threads(), t = omp_get_thread_num();
    const int c0 = (int)(cin * t / nt), c1 = (int)(cin * (t + 1) / nt);
    std::vector<double> dcol(cin);
    for (int64_t i = 0; c0 < c1 && i < n_out; ++i)
      for (int k = 0; k < K3; ++k) {
        int32_t j = nb[i * K3 + k];
        if (j < 0 || j >= n_in || (want && !want[j])) continue;
        for (int ci = c0; ci < c1; ++ci) {
          double acc = 0.0;
          const double* wk = w + ((int64_t)k * cin + ci) * cout;
          for (int co = 0; co < cout; ++co) acc += wk[co] * dy[i * cout + co];
          dcol[ci] = acc;
        }
        for (int ci = c0; ci < c1; ++ci) dx[j * cin + ci] += dcol[ci];
      }
  }
  return OK;
}

// Convolution backward w.r.t. the weights: dW = col^T . dY, i.e.
// dW[k][ci][co] = sum_i col[i][k*cin+ci] * dY[i][co].  entries (nullable):
// flat indices into [K^3][cin][cout] to compute, dw is then [nent].
int ocref_conv_bwd_weight(const int32_t* nb, int64_t n_out, int32_t K3, const double* x,
                          int64_t n_in, int32_t cin, const double* dy, int32_t cout,
                          const int64_t* entries, int64_t nent, double* dw) {
  if (!nb || !x || !dy || !dw || K3 < 1 || cin < 1 || cout < 1) return ERR_ARG;
  const int64_t total = (int64_t)K3 * cin * cout;
  if (entries) {
    for (int64_t e = 0; e < nent; ++e)
      if (entries[e] < 0 || entries[e] >= total) return ERR_ARG;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t e = 0; e < nent; ++e) {
      int64_t f = entries[e];
      int k = (int)(f / ((int64_t)cin * cout));
      int ci = (int)((f / cout) % cin);
      int co = (int)(f % cout);
      double acc = 0.0;
      for (int64_t i = 0; i < n_out; ++i) {
        int32_t j = nb[i * K3 + k];
        double c = (j >= 0 && j < n_in) ? x[j * cin + ci] : 0.0;
        acc += c * dy[i * cout + co];
      }
      dw[e] = acc;
    }
    return OK;
  }
#pragma omp parallel
  {
    std::vector<double> acc(cout);
#pragma omp for schedule(dynamic, 1)
    for (int64_t kc = 0; kc < (int64_t)K3 * cin; ++kc) {
      int k = (int)(kc / cin), ci = (int)(kc % cin);
      std::fill(acc.begin(), acc.end(), 0.0);
      for (int64_t i = 0; i < n_out; ++i) {
        int32_t j = nb[i * K3 + k];
        double c = (j >= 0 && j < n_in) ? x[j * cin + ci] : 0.0;
        if (c == 0.0) continue;
        for (int co = 0; co < cout; ++co) acc[co] += c * dy[i * cout + co];
      }
      for (int co = 0; co < cout; ++co) dw[kc * cout + co] = acc[co];
    }
  }
  return OK;
}

// Stride-2 renewal (Sec. 3.2; Fig. 2(d)): T_{l-1}[i] = Yhat[L_{l-1}[i]-1]
// if L_{l-1}[i] > 0, else 0.
int ocref_renew(const int32_t* labels, int64_t n_lm1, const double* yhat, int32_t c, double* y) {
  if (!labels || !yhat || !y || c < 1) return ERR_ARG;
  for (int64_t i = 0; i < n_lm1; ++i)
    for (int ch = 0; ch < c; ++ch)
      y[i * c + ch] = labels[i] > 0 ? yhat[(int64_t)(labels[i] - 1) * c + ch] : 0.0;
  return OK;
}

// Adjoint of the renewal: dYhat[L_{l-1}[i]-1] = dT_{l-1}[i] for L > 0.
int ocref_renew_bwd(const int32_t* labels, int64_t n_lm1, const double* dy, int32_t c, int64_t m,
                    double* dyhat) {
  if (!labels || !dy || !dyhat || c < 1) return ERR_ARG;
  std::fill(dyhat, dyhat + m * c, 0.0);
  for (int64_t i = 0; i < n_lm1; ++i)
    if (labels[i] > 0)
      for (int ch = 0; ch < c; ++ch) dyhat[(int64_t)(labels[i] - 1) * c + ch] = dy[i * c + ch];
  return OK;
}

// Max-pooling 2x2x2 (Sec. 3.2 "Pooling", Fig. 5): the max of every 8
// contiguous rows of depth l into That[g] (first maximum wins a tie; switch
// sw[g][ch] = its child index), then T_{l-1}[i] = That[L_{l-1}[i]-1] when
// L > 0, else 0.  n_l must be 8 * M_{l-1}.
int ocref_pool_fwd(const int32_t* labels, int64_t n_lm1, const double* x, int64_t n_l, int32_t c,
                   double* y, uint8_t* sw) {
  if (!labels || !x || !y || !sw || c < 1 || n_l % 8) return ERR_ARG;
  const int64_t m = n_l / 8;
  std::vector<double> that(m * c);
  for (int64_t g = 0; g < m; ++g)
    for (int ch = 0; ch < c; ++ch) {
      double best = x[(8 * g) * c + ch];
      int s = 0;
      for (int k = 1; k < 8; ++k) {
        double v = x[(8 * g + k) * c + ch];
        if (v > best) {
          best = v;
          s = k;
        }
      }
      that[g * c + ch] = best;
      sw[g * c + ch] = (uint8_t)s;
    }
  return ocref_renew(labels, n_lm1, that.data(), c, y);
}

// Max-pooling backward: the gradient of T_{l-1}[i] goes to the switch
// location of group L_{l-1}[i]-1; every other child gets zero.
int ocref_pool_bwd(const int32_t* labels, int64_t n_lm1, const double* dy, const uint8_t* sw,
                   int32_t c, int64_t n_l, double* dx) {
  if (!labels || !dy || !sw || !dx || c < 1) return ERR_ARG;
  std::fill(dx, dx + n_l * c, 0.0);
  for (int64_t i = 0; i < n_lm1; ++i) {
    if (labels[i] <= 0) continue;
    int64_t g = labels[i] - 1;
    for (int ch = 0; ch < c; ++ch) dx[(8 * g + sw[g * c + ch]) * c + ch] = dy[i * c + ch];
  }
  return OK;
}

// Max-unpooling (Sec. 3.2 "Unpooling", Fig. 5): T_{l-1}[i] is placed at the
// switch location among the 8 children of group L_{l-1}[i]-1; every other
// child is zero.  Rows of empty parents have no children and are dropped.
int ocref_unpool_fwd(const int32_t* labels, int64_t n_lm1, const double* x, const uint8_t* sw,
                     int32_t c, int64_t n_l, double* y) {
  return ocref_pool_bwd(labels, n_lm1, x, sw, c, n_l, y);
}

// Max-unpooling backward: dT_{l-1}[i] = dT_l[8g + sw[g]] for g = L-1, 0 for
// empty parents.
int ocref_unpool_bwd(const int32_t* labels, int64_t n_lm1, const double* dy, const uint8_t* sw,
                     int32_t c, double* dx) {
  if (!labels || !dy || !sw || !dx || c < 1) return ERR_ARG;
  for (int64_t i = 0; i < n_lm1; ++i)
    for (int ch = 0; ch < c; ++ch) {
      double v = 0.0;
      if (labels[i] > 0) {
        int64_t g = labels[i] - 1;
        v = dy[(8 * g + sw[g * c + ch]) * c + ch];
      }
      dx[i * c + ch] = v;
    }
  return OK;
}

// Threads the OpenMP loops above use (reported beside CPU timings).
int ocref_num_threads(void) { return omp_get_max_threads(); }

// Threads of the parallel loops that follow (n >= 1); timing only.
int ocref_set_num_threads(int32_t n) {
  if (n < 1) return 1;
  omp_set_num_threads(n);
  return 0;
}

// ReLU (Sec. 4): y = max(0, x); backward dx = dy * [x > 0].
int ocref_relu_fwd(const double* x, int64_t n, double* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = x[i] > 0.0 ? x[i] : 0.0;
  return OK;
}

int ocref_relu_bwd(const double* x, const double* dy, int64_t n, double* dx) {
  for (int64_t i = 0; i < n; ++i) dx[i] = x[i] > 0.0 ? dy[i] : 0.0;
  return OK;
}

}  // extern "C"
