// Sparse 3D convolution oracle: a plain, slow, CPU-only statement of what the
// method in "Sparse 3D convolutional neural networks" (Graham) computes.
//
// TEST INFRASTRUCTURE ONLY.  Only the tests, the package's smoke check and the
// benchmark's CPU-baseline leg may load this library.  It shares no code with
// the GPU library: no headers, kernels, tables or helpers.
//
// Everything is double precision.  Each function states the passage of the
// paper it follows (section 1.3 "Sparse operations" unless said otherwise).
//
// Readings taken where the paper is silent:
//  * the output extent is "valid": m_out = floor((m - f) / s) + 1 per axis,
//    as in Figure 3 (a 2x2 filter on a 6x6 grid gives a 5x5 output);
//  * output site o sees input sites s*o + k, k in [0, f)^3, offset index
//    k = (kz*f + ky)*f + kx;
//  * the tetrahedral lattice (section 1.2) is written in skewed integer
//    coordinates: a grid of size m is the sites x + y + z < m (equal extents
//    m on the three axes), a filter of size f the C(f+2, 3) offsets
//    kx + ky + kz < f, numbered in the cubic scan order above restricted to
//    those offsets, and output o is valid when its whole window lies in the
//    grid, i.e. ox + oy + oz < floor((m - f) / s) + 1;
//  * the 2D lattices of Figure 2 (i) and (ii) are the grids with mz = 1 and
//    z = 0: the square lattice takes the f^2 offsets (kx, ky, 0), the
//    triangular one (skewed coordinates, sites x + y < m, mx = my = m) the
//    C(f+1, 2) offsets kx + ky < f, with the same numbering and validity
//    rules as the 3D lattices;
//  * site key = ((b*mz + z)*my + y)*mx + x; output rows are numbered in
//    ascending key order starting at 0;
//  * W is stored offset-major: W[k][ci][co] (row k*Cin + ci of the
//    (f^3 n_in) x n_out matrix);
//  * an inactive input position inside a window contributes the ground state
//    g_in, both to the convolution (the rows of Q) and to max-pooling;
//  * max-pooling keeps the first strict maximum scanning k upwards;
//  * the hypercubic lattice in d = 1..4 dimensions (section 1.2: the same
//    construction in any dimension) takes sites (b, x_1, .., x_d) with key
//    ((b*m_d + x_d)*m_(d-1) + ..)*m_1 + x_1 and the f^d offsets numbered
//    k = sum_a k_a f^(a-1), k_1 fastest (in 3D the key and numbering above);
//  * gradients are those of the dense-equivalent function, for the loss
//    sum_active <dy[o], y[o]> + <dg_out, g_out>; ReLU'(0) = 0.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <map>
#include <set>
#include <vector>

namespace {

enum Status { OK = 0, INVALID = 1, RANGE = 2, DUPLICATE = 3, OVERFLOW_ = 4 };

struct Grid {
  int64_t B = 0, mx = 0, my = 0, mz = 0;
};

uint64_t key_of(const Grid& g, int64_t b, int64_t x, int64_t y, int64_t z) {
  return static_cast<uint64_t>(((b * g.mz + z) * g.my + y) * g.mx + x);
}

struct Rulebook {
  int f = 0, s = 0, K = 0;
  int lattice = 0;  // 0 cubic, 1 tetrahedral, 2 square, 3 triangular
  std::vector<int> offs;  // offset k -> (kz*f + ky)*f + kx of the cube scan
  Grid gin, gout;
  int64_t a_in = 0;
  // H_in: active input location -> row of M_in (the paper's map H_in).
  std::map<uint64_t, int32_t> H_in;
  // H_out: active output locations in ascending key order; row = index.
  std::vector<uint64_t> out_keys;
  std::vector<int32_t> out_coords;  // [a_out][4] = (b, x, y, z)
  // per filter offset k: (input row, output row), ordered by output row
  std::vector<std::vector<std::pair<int32_t, int32_t>>> lists;
  // hypercubic sites of D coordinates (orc_rb_build_nd): extents m_1..m_D of
  // the input and output grids; out_coords then has D + 1 entries per row
  bool nd = false;
  int D = 3;
  std::vector<int64_t> m_in, m_out;

  int64_t a_out() const { return static_cast<int64_t>(out_keys.size()); }

  // offset index -> (kx, ky, kz)
  void offset(int k, int64_t* kx, int64_t* ky, int64_t* kz) const {
    const int c = offs[k];
    *kx = c % f;
    *ky = (c / f) % f;
    *kz = c / (f * f);
  }

  // Row of M_in at input site s*o + k for output row o, or -1 when that site
  // is not active (then the window sees the ground state there).
  int32_t input_row(int64_t o, int k) const {
    if (nd) return input_row_nd(o, k);
    const int32_t* c = &out_coords[4 * o];
    int64_t kx, ky, kz;
    offset(k, &kx, &ky, &kz);
    uint64_t key = key_of(gin, c[0], s * c[1] + kx, s * c[2] + ky, s * c[3] + kz);
    auto it = H_in.find(key);
    return it == H_in.end() ? -1 : it->second;
  }

  // The same for the hypercubic sites of orc_rb_build_nd: input s*o + k.
  int32_t input_row_nd(int64_t o, int k) const;
};

int64_t out_extent(int64_t m, int f, int s) { return m >= f ? (m - f) / s + 1 : 0; }

// key of site (b, x_1..x_D) in extents m (x_1 fastest)
uint64_t key_nd(int64_t b, const int64_t* x, const std::vector<int64_t>& m, int D) {
  uint64_t key = static_cast<uint64_t>(b);
  for (int a = D - 1; a >= 0; --a) key = key * static_cast<uint64_t>(m[a]) + static_cast<uint64_t>(x[a]);
  return key;
}

// component a of offset k (k = sum_a k_a f^a)
int64_t offset_nd(int k, int a, int f) {
  int64_t v = k;
  for (int i = 0; i < a; ++i) v /= f;
  return v % f;
}

bool mul_ok(int64_t a, int64_t b, int64_t lim) { return a == 0 || b <= lim / a; }

int32_t Rulebook::input_row_nd(int64_t o, int k) const {
  const int32_t* c = &out_coords[(D + 1) * o];
  int64_t x[4] = {0, 0, 0, 0};
  for (int a = 0; a < D; ++a) x[a] = s * (int64_t)c[1 + a] + offset_nd(k, a, f);
  auto it = H_in.find(key_nd(c[0], x, m_in, D));
  return it == H_in.end() ? -1 : it->second;
}

}  // namespace

extern "C" {

// Step 1 of the convolution recipe: build H_in from the active sites, find the
// active output sites (an output is active iff some input site in its window is
// active, the second active-site rule of section 1.3) and number them; then list,
// per filter offset, which active input feeds which active output.  These lists
// are the non-ground-state blocks of the matrix Q of step 2.
int orc_rb_build_lattice(const int32_t* coords, int64_t n, const int64_t* grid, int32_t f,
                         int32_t s, int32_t lattice, void** out) {
  *out = nullptr;
  if (n < 0 || f < 1 || s < 1 || (n > 0 && coords == nullptr) || grid == nullptr) return INVALID;
  if (lattice < 0 || lattice > 3) return INVALID;
  const bool planar = lattice >= 2;                    // square, triangular
  const bool simplex = lattice == 1 || lattice == 3;   // tetrahedral, triangular
  Grid g{grid[0], grid[1], grid[2], grid[3]};
  if (g.B < 1 || g.mx < 1 || g.my < 1 || g.mz < 1) return INVALID;
  // a 2D grid has one z plane; a simplex grid has one size m: the sites
  // with coordinate sum below m
  if (planar && g.mz != 1) return INVALID;
  if (simplex && (g.my != g.mx || (!planar && g.mz != g.mx))) return INVALID;
  const int fz = planar ? 1 : f;  // filter extent along z
  const int64_t LIM = INT64_C(1) << 62;
  if (!mul_ok(g.B, g.mz, LIM) || !mul_ok(g.B * g.mz, g.my, LIM) ||
      !mul_ok(g.B * g.mz * g.my, g.mx, LIM))
    return OVERFLOW_;
  if (n > INT32_MAX) return OVERFLOW_;

  Rulebook* rb = new Rulebook();
  rb->f = f;
  rb->s = s;
  rb->lattice = lattice;
  for (int kz = 0; kz < fz; ++kz)
    for (int ky = 0; ky < f; ++ky)
      for (int kx = 0; kx < f; ++kx)
        if (!simplex || kx + ky + kz < f) rb->offs.push_back((kz * f + ky) * f + kx);
  rb->K = static_cast<int>(rb->offs.size());
  rb->gin = g;
  rb->gout = Grid{g.B, out_extent(g.mx, f, s), out_extent(g.my, f, s), out_extent(g.mz, fz, s)};
  rb->a_in = n;

  for (int64_t r = 0; r < n; ++r) {
    const int32_t* c = coords + 4 * r;
    if (c[0] < 0 || c[0] >= g.B || c[1] < 0 || c[1] >= g.mx || c[2] < 0 || c[2] >= g.my ||
        c[3] < 0 || c[3] >= g.mz ||
        (simplex && (int64_t)c[1] + c[2] + c[3] >= g.mx)) {
      delete rb;
      return RANGE;
    }
    uint64_t key = key_of(g, c[0], c[1], c[2], c[3]);
    if (!rb->H_in.emplace(key, static_cast<int32_t>(r)).second) {
      delete rb;
      return DUPLICATE;
    }
  }

  // Active outputs: every o with s*o + k equal to an active input for some k.
  const Grid& go = rb->gout;
  std::set<uint64_t> H_out;
  for (int64_t r = 0; r < n; ++r) {
    const int32_t* c = coords + 4 * r;
    for (int k = 0; k < rb->K; ++k) {
      int64_t kx, ky, kz;
      rb->offset(k, &kx, &ky, &kz);
      int64_t d[3] = {c[1] - kx, c[2] - ky, c[3] - kz};
      int64_t m[3] = {go.mx, go.my, go.mz};
      bool ok = true;
      for (int a = 0; a < 3; ++a)
        ok = ok && d[a] >= 0 && d[a] % s == 0 && d[a] / s < m[a];
      // simplex lattices: the output grid is the sites with coordinate sum below m_out
      if (simplex) ok = ok && (d[0] + d[1] + d[2]) / s < go.mx;
      if (ok) H_out.insert(key_of(go, c[0], d[0] / s, d[1] / s, d[2] / s));
    }
  }
  if (static_cast<int64_t>(H_out.size()) > INT32_MAX) {
    delete rb;
    return OVERFLOW_;
  }
  rb->out_keys.assign(H_out.begin(), H_out.end());
  rb->out_coords.resize(4 * rb->out_keys.size());
  for (size_t o = 0; o < rb->out_keys.size(); ++o) {
    uint64_t key = rb->out_keys[o];
    int64_t x = key % go.mx;
    key /= go.mx;
    int64_t y = key % go.my;
    key /= go.my;
    int64_t z = key % go.mz;
    int64_t b = key / go.mz;
    int32_t* c = &rb->out_coords[4 * o];
    c[0] = (int32_t)b;
    c[1] = (int32_t)x;
    c[2] = (int32_t)y;
    c[3] = (int32_t)z;
  }

  // Rule lists: for each output (ascending) and offset, the input row if active.
  rb->lists.assign(rb->K, {});
  int64_t total = 0;
  for (int64_t o = 0; o < rb->a_out(); ++o) {
    for (int k = 0; k < rb->K; ++k) {
      int32_t r = rb->input_row(o, k);
      if (r >= 0) {
        rb->lists[k].emplace_back(r, static_cast<int32_t>(o));
        ++total;
      }
    }
  }
  if (total > INT32_MAX) {
    delete rb;
    return OVERFLOW_;
  }
  *out = rb;
  return OK;
}

// The cubic lattice of the recipe above.
int orc_rb_build(const int32_t* coords, int64_t n, const int64_t* grid, int32_t f, int32_t s,
                 void** out) {
  return orc_rb_build_lattice(coords, n, grid, f, s, 0, out);
}

// Step 1 on the hypercubic lattice of D = 1..4 dimensions (section 1.2):
// sites (b, x_1..x_D), coords int32[n][D + 1], grid (B, m_1..m_D), f^D
// offsets.  The same three parts as above: H_in, the active outputs numbered
// in key order, the rule lists in output order.
int orc_rb_build_nd(const int32_t* coords, int64_t n, int32_t D, const int64_t* grid, int32_t f,
                    int32_t s, void** out) {
  *out = nullptr;
  if (n < 0 || f < 1 || s < 1 || D < 1 || D > 4 || (n > 0 && coords == nullptr) ||
      grid == nullptr)
    return INVALID;
  const int64_t B = grid[0];
  if (B < 1) return INVALID;
  const int64_t LIM = INT64_C(1) << 62;
  int64_t sites = B;
  for (int a = 0; a < D; ++a) {
    if (grid[1 + a] < 1) return INVALID;
    if (!mul_ok(sites, grid[1 + a], LIM)) return OVERFLOW_;
    sites *= grid[1 + a];
  }
  if (n > INT32_MAX) return OVERFLOW_;
  int64_t K = 1;
  for (int a = 0; a < D; ++a) K *= f;
  if (K > INT32_MAX) return OVERFLOW_;

  Rulebook* rb = new Rulebook();
  rb->nd = true;
  rb->D = D;
  rb->f = f;
  rb->s = s;
  rb->K = static_cast<int>(K);
  for (int k = 0; k < rb->K; ++k) rb->offs.push_back(k);
  for (int a = 0; a < D; ++a) {
    rb->m_in.push_back(grid[1 + a]);
    rb->m_out.push_back(out_extent(grid[1 + a], f, s));
  }
  rb->gin = Grid{B, 1, 1, 1};
  rb->gout = Grid{B, 1, 1, 1};
  rb->a_in = n;

  for (int64_t r = 0; r < n; ++r) {
    const int32_t* c = coords + (D + 1) * r;
    int64_t x[4] = {0, 0, 0, 0};
    bool ok = c[0] >= 0 && c[0] < B;
    for (int a = 0; a < D; ++a) {
      x[a] = c[1 + a];
      ok = ok && x[a] >= 0 && x[a] < rb->m_in[a];
    }
    if (!ok) {
      delete rb;
      return RANGE;
    }
    if (!rb->H_in.emplace(key_nd(c[0], x, rb->m_in, D), static_cast<int32_t>(r)).second) {
      delete rb;
      return DUPLICATE;
    }
  }

  // active outputs: every o with s*o + k an active input for some k
  std::set<uint64_t> H_out;
  for (int64_t r = 0; r < n; ++r) {
    const int32_t* c = coords + (D + 1) * r;
    for (int k = 0; k < rb->K; ++k) {
      int64_t o[4] = {0, 0, 0, 0};
      bool ok = true;
      for (int a = 0; a < D; ++a) {
        const int64_t d = c[1 + a] - offset_nd(k, a, f);
        ok = ok && d >= 0 && d % s == 0 && d / s < rb->m_out[a];
        o[a] = d / s;
      }
      if (ok) H_out.insert(key_nd(c[0], o, rb->m_out, D));
    }
  }
  if (static_cast<int64_t>(H_out.size()) > INT32_MAX) {
    delete rb;
    return OVERFLOW_;
  }
  rb->out_keys.assign(H_out.begin(), H_out.end());
  rb->out_coords.resize((D + 1) * rb->out_keys.size());
  for (size_t o = 0; o < rb->out_keys.size(); ++o) {
    uint64_t key = rb->out_keys[o];
    int32_t* c = &rb->out_coords[(D + 1) * o];
    for (int a = 0; a < D; ++a) {
      c[1 + a] = static_cast<int32_t>(key % static_cast<uint64_t>(rb->m_out[a]));
      key /= static_cast<uint64_t>(rb->m_out[a]);
    }
    c[0] = static_cast<int32_t>(key);
  }

  rb->lists.assign(rb->K, {});
  int64_t total = 0;
  for (int64_t o = 0; o < rb->a_out(); ++o)
    for (int k = 0; k < rb->K; ++k) {
      const int32_t r = rb->input_row(o, k);
      if (r >= 0) {
        rb->lists[k].push_back({r, static_cast<int32_t>(o)});
        ++total;
      }
    }
  if (total > INT32_MAX) {
    delete rb;
    return OVERFLOW_;
  }
  *out = rb;
  return OK;
}

// info = {a_in, a_out, n_pairs, K, D, B, m_out_1 .. m_out_4 (0 past D)}
void orc_rb_info_nd(const void* h, int64_t* info) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  int64_t np = 0;
  for (auto& l : rb->lists) np += (int64_t)l.size();
  info[0] = rb->a_in;
  info[1] = rb->a_out();
  info[2] = np;
  info[3] = rb->K;
  info[4] = rb->nd ? rb->D : 3;
  info[5] = rb->gout.B;
  const int64_t m3[3] = {rb->gout.mx, rb->gout.my, rb->gout.mz};
  for (int a = 0; a < 4; ++a)
    info[6 + a] = rb->nd ? (a < rb->D ? rb->m_out[a] : 0) : (a < 3 ? m3[a] : 0);
}

void orc_rb_free(void* h) { delete static_cast<Rulebook*>(h); }

// info = {a_in, a_out, n_pairs, K, B, mx_out, my_out, mz_out}
void orc_rb_info(const void* h, int64_t* info) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  int64_t np = 0;
  for (auto& l : rb->lists) np += (int64_t)l.size();
  info[0] = rb->a_in;
  info[1] = rb->a_out();
  info[2] = np;
  info[3] = rb->K;
  info[4] = rb->gout.B;
  info[5] = rb->gout.mx;
  info[6] = rb->gout.my;
  info[7] = rb->gout.mz;
}

// off[K+1]: list k occupies pair positions [off[k], off[k+1]).
void orc_rb_offsets(const void* h, int64_t* off) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  off[0] = 0;
  for (int k = 0; k < rb->K; ++k) off[k + 1] = off[k] + (int64_t)rb->lists[k].size();
}

void orc_rb_export(const void* h, int32_t* out_coords, int32_t* in_rows, int32_t* out_rows) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  if (out_coords && !rb->out_coords.empty())
    std::memcpy(out_coords, rb->out_coords.data(), rb->out_coords.size() * sizeof(int32_t));
  int64_t p = 0;
  for (auto& l : rb->lists)
    for (auto& pr : l) {
      if (in_rows) in_rows[p] = pr.first;
      if (out_rows) out_rows[p] = pr.second;
      ++p;
    }
}

// Ground state of a convolution's output (section 1.3: inactive sites all hold
// the same vector, which can be computed in advance).  An output site whose
// window is entirely inactive sees g_in at every offset, so
// g_out = act(B + sum_k g_in W_k).
static void conv_ground_pre(const Rulebook* rb, const double* g_in, const double* W,
                            const double* bias, int Cin, int Cout, std::vector<double>& gpre) {
  gpre.assign(Cout, 0.0);
  for (int co = 0; co < Cout; ++co) gpre[co] = bias ? bias[co] : 0.0;
  for (int k = 0; k < rb->K; ++k)
    for (int ci = 0; ci < Cin; ++ci)
      for (int co = 0; co < Cout; ++co)
        gpre[co] += g_in[ci] * W[((int64_t)k * Cin + ci) * Cout + co];
}

// Steps 2 and 3 of the convolution recipe, literally: row o of Q concatenates,
// over the filter offsets k, the vector at input site s*o + k (a row of M_in
// when active, else g_in); M_out = Q W + B.  ReLU is applied when relu != 0.
// rows == nullptr computes every output row into y[a_out][Cout]; otherwise only
// output rows rows[0..nrows) into y[nrows][Cout].
int orc_conv_fwd(const void* h, const double* x, const double* g_in, const double* W,
                 const double* bias, int32_t Cin, int32_t Cout, int32_t relu,
                 const int64_t* rows, int64_t nrows, double* y, double* g_out) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  if (Cin < 1 || Cout < 1) return INVALID;
  int64_t count = rows ? nrows : rb->a_out();
  std::vector<double> q(Cin);
  for (int64_t j = 0; j < count; ++j) {
    int64_t o = rows ? rows[j] : j;
    if (o < 0 || o >= rb->a_out()) return RANGE;
    double* yo = y + j * Cout;
    for (int co = 0; co < Cout; ++co) yo[co] = bias ? bias[co] : 0.0;
    for (int k = 0; k < rb->K; ++k) {
      int32_t r = rb->input_row(o, k);
      for (int ci = 0; ci < Cin; ++ci) q[ci] = r >= 0 ? x[(int64_t)r * Cin + ci] : g_in[ci];
      for (int ci = 0; ci < Cin; ++ci)
        for (int co = 0; co < Cout; ++co) yo[co] += q[ci] * W[((int64_t)k * Cin + ci) * Cout + co];
    }
    if (relu)
      for (int co = 0; co < Cout; ++co) yo[co] = yo[co] > 0.0 ? yo[co] : 0.0;
  }
  if (g_out) {
    std::vector<double> gpre;
    conv_ground_pre(rb, g_in, W, bias, Cin, Cout, gpre);
    for (int co = 0; co < Cout; ++co) g_out[co] = relu ? (gpre[co] > 0.0 ? gpre[co] : 0.0) : gpre[co];
  }
  return OK;
}

// Gradients of the convolution above (the paper trains these networks but does
// not spell out the backward pass; this is the derivative of the same
// dense-equivalent function).  Loss = sum_o <dy[o], y[o]> + <dg_out, g_out>.
// Any output pointer may be null.  Outputs are overwritten.
int orc_conv_bwd(const void* h, const double* x, const double* g_in, const double* W,
                 const double* bias, const double* dy, const double* dg_out, int32_t Cin,
                 int32_t Cout, int32_t relu, double* dx, double* dg_in, double* dW,
                 double* dbias) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  if (Cin < 1 || Cout < 1) return INVALID;
  const int K = rb->K;
  const int64_t a_out = rb->a_out();
  std::vector<double> gpre;
  conv_ground_pre(rb, g_in, W, bias, Cin, Cout, gpre);
  // gradient reaching the ground-state pre-activation
  std::vector<double> dgb(Cout, 0.0);
  for (int co = 0; co < Cout; ++co) {
    double d = dg_out ? dg_out[co] : 0.0;
    dgb[co] = (relu && !(gpre[co] > 0.0)) ? 0.0 : d;
  }
  std::vector<double> gx(rb->a_in * (int64_t)Cin, 0.0), gg(Cin, 0.0),
      gW((int64_t)K * Cin * Cout, 0.0), gB(Cout, 0.0);
  std::vector<double> pre(Cout), dyb(Cout), q(Cin);
  for (int64_t o = 0; o < a_out; ++o) {
    // recompute the pre-activation for the ReLU mask
    if (relu) {
      for (int co = 0; co < Cout; ++co) pre[co] = bias ? bias[co] : 0.0;
      for (int k = 0; k < K; ++k) {
        int32_t r = rb->input_row(o, k);
        for (int ci = 0; ci < Cin; ++ci) {
          double v = r >= 0 ? x[(int64_t)r * Cin + ci] : g_in[ci];
          for (int co = 0; co < Cout; ++co) pre[co] += v * W[((int64_t)k * Cin + ci) * Cout + co];
        }
      }
    }
    for (int co = 0; co < Cout; ++co) {
      double d = dy[o * Cout + co];
      dyb[co] = (relu && !(pre[co] > 0.0)) ? 0.0 : d;
      gB[co] += dyb[co];
    }
    for (int k = 0; k < K; ++k) {
      int32_t r = rb->input_row(o, k);
      for (int ci = 0; ci < Cin; ++ci) q[ci] = r >= 0 ? x[(int64_t)r * Cin + ci] : g_in[ci];
      for (int ci = 0; ci < Cin; ++ci) {
        const double* Wk = W + ((int64_t)k * Cin + ci) * Cout;
        double* gWk = gW.data() + ((int64_t)k * Cin + ci) * Cout;
        double back = 0.0;
        for (int co = 0; co < Cout; ++co) {
          gWk[co] += q[ci] * dyb[co];
          back += Wk[co] * dyb[co];
        }
        if (r >= 0)
          gx[(int64_t)r * Cin + ci] += back;
        else
          gg[ci] += back;
      }
    }
  }
  // ground-state path: g_pre = B + sum_k g_in W_k
  for (int co = 0; co < Cout; ++co) gB[co] += dgb[co];
  for (int k = 0; k < K; ++k)
    for (int ci = 0; ci < Cin; ++ci)
      for (int co = 0; co < Cout; ++co) {
        int64_t w = ((int64_t)k * Cin + ci) * Cout + co;
        gW[w] += g_in[ci] * dgb[co];
        gg[ci] += W[w] * dgb[co];
      }
  if (dx) std::copy(gx.begin(), gx.end(), dx);
  if (dg_in) std::copy(gg.begin(), gg.end(), dg_in);
  if (dW) std::copy(gW.begin(), gW.end(), dW);
  if (dbias) std::copy(gB.begin(), gB.end(), dbias);
  return OK;
}

// Max-pooling "is similar" to the convolution (end of section 1.3): output o
// takes, per channel, the maximum over the f^3 positions of its window, each
// position holding a row of M_in when active and g_in otherwise.  arg_k[o][c]
// receives the winning offset and arg_inactive[o][c] = 1 when that position was
// inactive.  g_out = g_in (a window with no active site sees only g_in).
int orc_maxpool_fwd(const void* h, const double* x, const double* g_in, int32_t C, double* y,
                    double* g_out, int32_t* arg_k, uint8_t* arg_inactive) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  if (C < 1) return INVALID;
  for (int64_t o = 0; o < rb->a_out(); ++o) {
    std::vector<int32_t> r(rb->K);
    for (int k = 0; k < rb->K; ++k) r[k] = rb->input_row(o, k);
    for (int c = 0; c < C; ++c) {
      double best = 0.0;
      int bk = -1;
      for (int k = 0; k < rb->K; ++k) {
        double v = r[k] >= 0 ? x[(int64_t)r[k] * C + c] : g_in[c];
        if (bk < 0 || v > best) {
          best = v;
          bk = k;
        }
      }
      y[o * C + c] = best;
      if (arg_k) arg_k[o * C + c] = bk;
      if (arg_inactive) arg_inactive[o * C + c] = r[bk] < 0 ? 1 : 0;
    }
  }
  if (g_out)
    for (int c = 0; c < C; ++c) g_out[c] = g_in[c];
  return OK;
}

// Gradient of the max-pooling above: dy[o][c] flows to the winning position;
// a winning inactive position passes it to the ground state, and g_out = g_in
// passes dg_out through unchanged.
int orc_maxpool_bwd(const void* h, const double* x, const double* g_in, const double* dy,
                    const double* dg_out, int32_t C, double* dx, double* dg_in) {
  const Rulebook* rb = static_cast<const Rulebook*>(h);
  if (C < 1) return INVALID;
  int64_t a_out = rb->a_out();
  std::vector<double> y(a_out * (int64_t)C);
  std::vector<int32_t> ak(a_out * (int64_t)C);
  orc_maxpool_fwd(h, x, g_in, C, y.data(), nullptr, ak.data(), nullptr);
  std::vector<double> gx(rb->a_in * (int64_t)C, 0.0), gg(C, 0.0);
  for (int c = 0; c < C; ++c) gg[c] = dg_out ? dg_out[c] : 0.0;
  for (int64_t o = 0; o < a_out; ++o)
    for (int c = 0; c < C; ++c) {
      int k = ak[o * C + c];
      int32_t r = rb->input_row(o, k);
      if (r >= 0)
        gx[(int64_t)r * C + c] += dy[o * C + c];
      else
        gg[c] += dy[o * C + c];
    }
  if (dx) std::copy(gx.begin(), gx.end(), dx);
  if (dg_in) std::copy(gg.begin(), gg.end(), dg_in);
  return OK;
}

}  // extern "C"
