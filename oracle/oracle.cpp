/*
 * CPU oracle for the Polyglot window-ranking language model SGD step.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * reference that the GPU library is checked against.  Only the test suite,
 * the package smoke check and the CPU-baseline leg of the benchmark may load
 * it.  It shares no code, header, table or helper with the HIP library, and
 * the HIP library never calls it.
 *
 * What is computed, and where it comes from
 * -----------------------------------------
 * The paper (Kulkarni, Al-Rfou, Perozzi, Skiena: "Exploring the power of
 * GPU's for training Polyglot language models", arXiv:1404.1521) trains the
 * Polyglot language model, which it describes as close to the SENNA
 * ranking language model (§1 Introduction), with minibatch SGD in Theano
 * (§2 Experimental Setup; minibatch size, §4.6).  The paper does not write
 * the model out.  The reading adopted here is the SENNA-style window ranker:
 *
 *   x      = concat(E[w_0], ..., E[w_{win-1}])            (K = win*d values)
 *   x~     = x with block c = win/2 replaced by E[corrupt] (centre corrupted)
 *   s(x)   = w2 . tanh(W1 x + b1) + b2                    (W1 is H x K)
 *   loss_b = max(0, 1 - s(x) + s(x~))                     (hinge ranking)
 *   L      = (1/B) sum_b loss_b                           (mean over batch)
 *
 * One step takes every gradient at the pre-step parameters, then applies
 * P <- P - lr * dL/dP to E, W1, b1, w2 and b2.  The embedding gradient is a
 * row scatter-add in which repeated rows accumulate: exactly the
 * "advanced indexing" increment W[I[k]] += Y[k] that §4.2 (Table 1,
 * GpuAdvancedIncSubtensor1) identifies as the hot spot and §4.3 optimises.
 *
 * Readings where the paper is silent (each also listed in the design notes):
 *   - hinge derivative at margin exactly 0 is taken as 0 (strict "> 0");
 *   - the loss is the batch mean, so gradients carry a 1/B factor;
 *   - a corrupt id equal to the true centre is not resampled (its gradient
 *     cancels analytically);
 *   - centre position c = win/2 (win odd), no padding tokens.
 *
 * Arithmetic: every floating-point operation is done in double.  Storage is
 * a template parameter S: S = double gives a pure float64 model (used by the
 * finite-difference and closed-form pins); S = float keeps parameters in
 * float32 storage, as the GPU library does, computes in double and rounds
 * once when a parameter is written back.
 *
 * Error contract: every entry point returns 0 on success or a negative code
 * (ORACLE_E*) and, on error, leaves every output untouched.
 */
#include <cmath>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <vector>
#include <algorithm>

namespace {

enum {
  ORACLE_OK = 0,
  ORACLE_EINVAL = -1,  /* bad dimension, even window, non-finite lr */
  ORACLE_ENULL = -2,   /* required pointer is NULL */
  ORACLE_EID = -5      /* an id is outside [0, V) */
};

struct Shape {
  int V, d, win, H, B;
  int K() const { return win * d; }
  int c() const { return win / 2; }
};

int check_shape(const Shape& s) {
  if (s.V <= 0 || s.d <= 0 || s.win <= 0 || s.H <= 0 || s.B < 0) return ORACLE_EINVAL;
  if (s.win % 2 == 0) return ORACLE_EINVAL;
  return ORACLE_OK;
}

int check_ids(const Shape& s, const int32_t* windows, const int32_t* corrupt) {
  for (long i = 0; i < (long)s.B * s.win; ++i)
    if (windows[i] < 0 || windows[i] >= s.V) return ORACLE_EID;
  if (corrupt)
    for (int b = 0; b < s.B; ++b)
      if (corrupt[b] < 0 || corrupt[b] >= s.V) return ORACLE_EID;
  return ORACLE_OK;
}

/* Builds the concatenated window vector x (length K) in double. */
template <typename S>
void build_window(const Shape& s, const S* E, const int32_t* ids, std::vector<double>& x) {
  for (int j = 0; j < s.win; ++j)
    for (int t = 0; t < s.d; ++t)
      x[(size_t)j * s.d + t] = (double)E[(size_t)ids[j] * s.d + t];
}

/* Forward pass of one window: z = W1 x + b1, h = tanh(z), returns s = w2.h + b2.
   The dot product runs over k in ascending order. */
template <typename S>
double forward(const Shape& s, const S* W1, const S* b1, const S* w2, const S* b2,
               const std::vector<double>& x, std::vector<double>& h) {
  const int K = s.K();
  double score = (double)b2[0];
  for (int i = 0; i < s.H; ++i) {
    double z = (double)b1[i];
    for (int k = 0; k < K; ++k) z += (double)W1[(size_t)i * K + k] * x[k];
    h[i] = std::tanh(z);
    score += (double)w2[i] * h[i];
  }
  return score;
}

/* Gradient accumulators of one step, all in double.  The embedding gradient
   is kept sparse: slot_of[row] is the slot of a touched row or -1, rows[] the
   touched rows in first-touch order, dE the slot-major gradient rows. */
struct Grads {
  std::vector<double> dW1, db1, dw2;
  double db2 = 0.0;
  std::vector<int> slot_of;
  std::vector<int32_t> rows;
  std::vector<double> dE;
  int d;
  Grads(const Shape& s) : dW1((size_t)s.H * s.K(), 0.0), db1(s.H, 0.0), dw2(s.H, 0.0),
                          slot_of(s.V, -1), d(s.d) {}
  double* row(int32_t r) {
    if (slot_of[r] < 0) {
      slot_of[r] = (int)rows.size();
      rows.push_back(r);
      dE.resize(dE.size() + d, 0.0);
    }
    return &dE[(size_t)slot_of[r] * d];
  }
};

/* Loss and gradients of the mean hinge ranking loss at the given parameters.
   Returns the summed (not yet averaged) hinge loss. */
template <typename S>
double loss_and_grads(const Shape& s, const S* E, const S* W1, const S* b1, const S* w2,
                      const S* b2, const int32_t* windows, const int32_t* corrupt,
                      Grads* g) {
  const int K = s.K(), c = s.c(), d = s.d, H = s.H;
  std::vector<double> x(K), xt(K), h(H), ht(H), dz(H), dzt(H), dx(K), dxt(K);
  double total = 0.0;
  for (int b = 0; b < s.B; ++b) {
    const int32_t* ids = windows + (size_t)b * s.win;
    /* true window and the copy whose centre word is corrupted */
    build_window(s, E, ids, x);
    xt = x;
    for (int t = 0; t < d; ++t) xt[(size_t)c * d + t] = (double)E[(size_t)corrupt[b] * d + t];

    const double sc = forward(s, W1, b1, w2, b2, x, h);
    const double sct = forward(s, W1, b1, w2, b2, xt, ht);
    const double margin = 1.0 - sc + sct;
    if (!(margin > 0.0)) continue; /* hinge inactive: no loss, zero gradient */
    total += margin;
    if (!g) continue;

    /* d(mean loss)/ds = -1/B, d(mean loss)/ds~ = +1/B */
    const double gs = -1.0 / s.B, gst = 1.0 / s.B;
    for (int i = 0; i < H; ++i) {
      g->dw2[i] += gs * h[i] + gst * ht[i];
      dz[i] = gs * (double)w2[i] * (1.0 - h[i] * h[i]);
      dzt[i] = gst * (double)w2[i] * (1.0 - ht[i] * ht[i]);
      g->db1[i] += dz[i] + dzt[i];
    }
    g->db2 += gs + gst;
    for (int i = 0; i < H; ++i)
      for (int k = 0; k < K; ++k)
        g->dW1[(size_t)i * K + k] += dz[i] * x[k] + dzt[i] * xt[k];

    /* input gradients dx = W1^T dz, dx~ = W1^T dz~ */
    for (int k = 0; k < K; ++k) {
      double a = 0.0, at = 0.0;
      for (int i = 0; i < H; ++i) {
        a += (double)W1[(size_t)i * K + k] * dz[i];
        at += (double)W1[(size_t)i * K + k] * dzt[i];
      }
      dx[k] = a;
      dxt[k] = at;
    }
    /* route them to embedding rows; repeated rows accumulate */
    for (int j = 0; j < s.win; ++j) {
      if (j == c) continue;
      double* r = g->row(ids[j]);
      for (int t = 0; t < d; ++t) r[t] += dx[(size_t)j * d + t] + dxt[(size_t)j * d + t];
    }
    {
      double* r = g->row(ids[c]);
      for (int t = 0; t < d; ++t) r[t] += dx[(size_t)c * d + t];
    }
    {
      double* r = g->row(corrupt[b]);
      for (int t = 0; t < d; ++t) r[t] += dxt[(size_t)c * d + t];
    }
  }
  return total;
}

template <typename S>
int train_step(const Shape& s, S* E, S* W1, S* b1, S* w2, S* b2, const int32_t* windows,
               const int32_t* corrupt, double lr, double* loss_out) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (!E || !W1 || !b1 || !w2 || !b2 || (s.B > 0 && (!windows || !corrupt))) return ORACLE_ENULL;
  if (!std::isfinite(lr)) return ORACLE_EINVAL;
  if (s.B == 0) return ORACLE_EINVAL;
  rc = check_ids(s, windows, corrupt);
  if (rc) return rc;

  Grads g(s);
  const double total = loss_and_grads(s, E, W1, b1, w2, b2, windows, corrupt, &g);

  /* SGD update with the gradients taken at the pre-step parameters */
  const size_t nW1 = (size_t)s.H * s.K();
  for (size_t q = 0; q < nW1; ++q) W1[q] = (S)((double)W1[q] - lr * g.dW1[q]);
  for (int i = 0; i < s.H; ++i) {
    b1[i] = (S)((double)b1[i] - lr * g.db1[i]);
    w2[i] = (S)((double)w2[i] - lr * g.dw2[i]);
  }
  b2[0] = (S)((double)b2[0] - lr * g.db2);
  for (size_t u = 0; u < g.rows.size(); ++u) {
    S* er = E + (size_t)g.rows[u] * s.d;
    const double* gr = &g.dE[u * s.d];
    for (int t = 0; t < s.d; ++t) er[t] = (S)((double)er[t] - lr * gr[t]);
  }
  if (loss_out) *loss_out = total / s.B;
  return ORACLE_OK;
}

template <typename S>
int gradients(const Shape& s, const S* E, const S* W1, const S* b1, const S* w2, const S* b2,
              const int32_t* windows, const int32_t* corrupt, double* loss, double* dE,
              double* dW1, double* db1, double* dw2, double* db2) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (s.B == 0) return ORACLE_EINVAL;
  if (!E || !W1 || !b1 || !w2 || !b2 || !windows || !corrupt) return ORACLE_ENULL;
  rc = check_ids(s, windows, corrupt);
  if (rc) return rc;
  Grads g(s);
  const double total = loss_and_grads(s, E, W1, b1, w2, b2, windows, corrupt, &g);
  if (loss) *loss = total / s.B;
  if (dE) {
    std::memset(dE, 0, sizeof(double) * (size_t)s.V * s.d);
    for (size_t u = 0; u < g.rows.size(); ++u)
      for (int t = 0; t < s.d; ++t) dE[(size_t)g.rows[u] * s.d + t] = g.dE[u * s.d + t];
  }
  if (dW1) std::memcpy(dW1, g.dW1.data(), sizeof(double) * g.dW1.size());
  if (db1) std::memcpy(db1, g.db1.data(), sizeof(double) * s.H);
  if (dw2) std::memcpy(dw2, g.dw2.data(), sizeof(double) * s.H);
  if (db2) *db2 = g.db2;
  return ORACLE_OK;
}

template <typename S>
int score(const Shape& s, const S* E, const S* W1, const S* b1, const S* w2, const S* b2,
          const int32_t* windows, double* out) {
  int rc = check_shape(s);
  if (rc) return rc;
  if (!E || !W1 || !b1 || !w2 || !b2 || (s.B > 0 && (!windows || !out))) return ORACLE_ENULL;
  rc = check_ids(s, windows, nullptr);
  if (rc) return rc;
  std::vector<double> x(s.K()), h(s.H);
  for (int b = 0; b < s.B; ++b) {
    build_window(s, E, windows + (size_t)b * s.win, x);
    out[b] = forward(s, W1, b1, w2, b2, x, h);
  }
  return ORACLE_OK;
}

/* The advanced-indexing increment of §4.2/§4.3: for k = 0..N-1 in order,
   table[idx[k]] += alpha * Y[k].  Each touched row is carried in double from
   its stored value through every increment in k order and rounded to the
   storage type once at the end. */
template <typename S>
int scatter_add(int rows, int d, S* table, const int32_t* idx, const S* Y, long N, double alpha) {
  if (rows <= 0 || d <= 0 || N < 0) return ORACLE_EINVAL;
  if (!std::isfinite(alpha)) return ORACLE_EINVAL;
  if (N > 0 && (!table || !idx || !Y)) return ORACLE_ENULL;
  for (long k = 0; k < N; ++k)
    if (idx[k] < 0 || idx[k] >= rows) return ORACLE_EID;
  std::vector<int> slot_of(rows, -1);
  std::vector<int32_t> touched;
  std::vector<double> acc;
  for (long k = 0; k < N; ++k) {
    const int32_t r = idx[k];
    if (slot_of[r] < 0) {
      slot_of[r] = (int)touched.size();
      touched.push_back(r);
      for (int t = 0; t < d; ++t) acc.push_back((double)table[(size_t)r * d + t]);
    }
    double* a = &acc[(size_t)slot_of[r] * d];
    for (int t = 0; t < d; ++t) a[t] += alpha * (double)Y[(size_t)k * d + t];
  }
  for (size_t u = 0; u < touched.size(); ++u)
    for (int t = 0; t < d; ++t) table[(size_t)touched[u] * d + t] = (S)acc[u * d + t];
  return ORACLE_OK;
}

/* ---- The general advanced-indexing op (§4.3 names it; the library form
   the paper contributes takes any table, any index vector and either an
   increment or an assignment).  Storage formats: IEEE binary32, bfloat16
   (the upper half of a binary32: 8 significant bits, binary32's exponent
   range) and IEEE binary16 (11 significant bits, exponents -14..15).
   Decoding is exact; encoding rounds the double to nearest, ties to even,
   in one step (no intermediate binary32). */
enum { ORACLE_F32 = 0, ORACLE_BF16 = 1, ORACLE_F16 = 2 };
enum { ORACLE_OP_INC = 0, ORACLE_OP_SET = 1 };

/* x rounded to p significant bits with the exponent of the leading bit
   clamped below at emin (gradual underflow) and overflow to infinity above
   2^(emax+1); the default rounding mode is to nearest, ties to even. */
double round_to_format(double x, int p, int emin, int emax) {
  if (x == 0.0 || !std::isfinite(x)) return x;
  int e;
  std::frexp(x, &e);  // |x| in [2^(e-1), 2^e)
  const int lead = std::max(e - 1, emin);
  const double q = std::ldexp(1.0, lead - (p - 1));  // spacing of the format at x
  const double r = std::nearbyint(x / q) * q;        // both scalings are exact
  if (std::fabs(r) >= std::ldexp(1.0, emax + 1)) return std::copysign(INFINITY, x);
  return r;
}

double decode_elem(const void* base, size_t i, int dtype) {
  if (dtype == ORACLE_F32) return (double)static_cast<const float*>(base)[i];
  const uint16_t h = static_cast<const uint16_t*>(base)[i];
  if (dtype == ORACLE_BF16) {
    const uint32_t u = (uint32_t)h << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return (double)f;
  }
  const int sign = h >> 15, ex = (h >> 10) & 31, man = h & 1023;
  double v;
  if (ex == 0) v = std::ldexp((double)man, -24);
  else if (ex == 31) v = man ? NAN : INFINITY;
  else v = std::ldexp(1.0 + man / 1024.0, ex - 15);
  return sign ? -v : v;
}

void encode_elem(void* base, size_t i, int dtype, double x) {
  if (dtype == ORACLE_F32) {
    static_cast<float*>(base)[i] = (float)round_to_format(x, 24, -126, 127);
    return;
  }
  uint16_t h;
  if (dtype == ORACLE_BF16) {
    const float f = std::isnan(x) ? NAN : (float)round_to_format(x, 8, -126, 127);  // exact
    uint32_t u;
    std::memcpy(&u, &f, 4);
    h = std::isnan(x) ? (uint16_t)0x7fc0 : (uint16_t)(u >> 16);
  } else {
    const double r = std::isnan(x) ? x : round_to_format(x, 11, -14, 15);
    const uint16_t sign = std::signbit(r) ? 0x8000 : 0;
    const double a = std::fabs(r);
    if (std::isnan(r)) h = 0x7e00;
    else if (std::isinf(r)) h = sign | 0x7c00;
    else if (a < std::ldexp(1.0, -14)) h = sign | (uint16_t)(a * std::ldexp(1.0, 24));  // subnormal or 0
    else {
      int e;
      std::frexp(a, &e);
      const int ex = e - 1 + 15;
      const uint16_t man = (uint16_t)((a / std::ldexp(1.0, e - 1) - 1.0) * 1024.0);
      h = sign | (uint16_t)(ex << 10) | man;
    }
  }
  static_cast<uint16_t*>(base)[i] = h;
}

/* op = inc: for k in order, table[idx[k]] += alpha * Y[k], each touched row
   carried in double from its stored value and rounded to the storage format
   once at the end.  op = set: for k in order, table[idx[k]] = Y[k] (the
   last entry of a row wins; alpha is unused).  Indices are int32 or int64;
   any index outside [0, rows) rejects the whole call before a write. */
int scatter_add_ex(int rows, int d, void* table, int dtype, const void* idx, int idx_bytes,
                   const void* Y, long N, double alpha, int op) {
  if (rows <= 0 || d <= 0 || N < 0) return ORACLE_EINVAL;
  if (dtype < ORACLE_F32 || dtype > ORACLE_F16 || (idx_bytes != 4 && idx_bytes != 8))
    return ORACLE_EINVAL;
  if (op != ORACLE_OP_INC && op != ORACLE_OP_SET) return ORACLE_EINVAL;
  if (op == ORACLE_OP_INC && !std::isfinite(alpha)) return ORACLE_EINVAL;
  if (N > 0 && (!table || !idx || !Y)) return ORACLE_ENULL;
  std::vector<int64_t> id(N);
  for (long k = 0; k < N; ++k) {
    id[k] = idx_bytes == 4 ? (int64_t) static_cast<const int32_t*>(idx)[k]
                           : static_cast<const int64_t*>(idx)[k];
    if (id[k] < 0 || id[k] >= rows) return ORACLE_EID;
  }
  if (op == ORACLE_OP_SET) {
    const size_t es = dtype == ORACLE_F32 ? 4 : 2;
    for (long k = 0; k < N; ++k)
      std::memcpy(static_cast<char*>(table) + (size_t)id[k] * d * es,
                  static_cast<const char*>(Y) + (size_t)k * d * es, d * es);
    return ORACLE_OK;
  }
  std::vector<long> slot_of(rows, -1);
  std::vector<int64_t> touched;
  std::vector<double> acc;
  for (long k = 0; k < N; ++k) {
    const int64_t r = id[k];
    if (slot_of[r] < 0) {
      slot_of[r] = (long)touched.size();
      touched.push_back(r);
      for (int t = 0; t < d; ++t) acc.push_back(decode_elem(table, (size_t)r * d + t, dtype));
    }
    double* a = &acc[(size_t)slot_of[r] * d];
    for (int t = 0; t < d; ++t) a[t] += alpha * decode_elem(Y, (size_t)k * d + t, dtype);
  }
  for (size_t u = 0; u < touched.size(); ++u)
    for (int t = 0; t < d; ++t) encode_elem(table, (size_t)touched[u] * d + t, dtype, acc[u * d + t]);
  return ORACLE_OK;
}

}  // namespace

extern "C" {

int oracle_scatter_add_ex(int rows, int d, void* table, int dtype, const void* idx, int idx_bytes,
                          const void* Y, long N, double alpha, int op) {
  return scatter_add_ex(rows, d, table, dtype, idx, idx_bytes, Y, N, alpha, op);
}

/* the storage formats' rounding alone, for pinning against other
   implementations: n doubles encoded into `out` (binary32 or 16-bit words) */
int oracle_encode(int dtype, const double* x, long n, void* out) {
  if (dtype < ORACLE_F32 || dtype > ORACLE_F16 || n < 0) return ORACLE_EINVAL;
  for (long i = 0; i < n; ++i) encode_elem(out, (size_t)i, dtype, x[i]);
  return ORACLE_OK;
}

int oracle_decode(int dtype, const void* in, long n, double* x) {
  if (dtype < ORACLE_F32 || dtype > ORACLE_F16 || n < 0) return ORACLE_EINVAL;
  for (long i = 0; i < n; ++i) x[i] = decode_elem(in, (size_t)i, dtype);
  return ORACLE_OK;
}

int oracle_train_step_f32(int V, int d, int win, int H, int B, float* E, float* W1, float* b1,
                          float* w2, float* b2, const int32_t* windows, const int32_t* corrupt,
                          double lr, double* loss) {
  return train_step<float>(Shape{V, d, win, H, B}, E, W1, b1, w2, b2, windows, corrupt, lr, loss);
}

int oracle_train_step_f64(int V, int d, int win, int H, int B, double* E, double* W1, double* b1,
                          double* w2, double* b2, const int32_t* windows, const int32_t* corrupt,
                          double lr, double* loss) {
  return train_step<double>(Shape{V, d, win, H, B}, E, W1, b1, w2, b2, windows, corrupt, lr, loss);
}

/* Loss and full gradients in float64 storage; dE is dense [V][d] (small V only). */
int oracle_gradients_f64(int V, int d, int win, int H, int B, const double* E, const double* W1,
                         const double* b1, const double* w2, const double* b2,
                         const int32_t* windows, const int32_t* corrupt, double* loss, double* dE,
                         double* dW1, double* db1, double* dw2, double* db2) {
  return gradients<double>(Shape{V, d, win, H, B}, E, W1, b1, w2, b2, windows, corrupt, loss, dE,
                           dW1, db1, dw2, db2);
}

/* Mean hinge loss only (no gradient), float64 storage. */
int oracle_loss_f64(int V, int d, int win, int H, int B, const double* E, const double* W1,
                    const double* b1, const double* w2, const double* b2, const int32_t* windows,
                    const int32_t* corrupt, double* loss) {
  Shape s{V, d, win, H, B};
  int rc = check_shape(s);
  if (rc) return rc;
  if (B == 0) return ORACLE_EINVAL;
  if (!E || !W1 || !b1 || !w2 || !b2 || !windows || !corrupt || !loss) return ORACLE_ENULL;
  rc = check_ids(s, windows, corrupt);
  if (rc) return rc;
  *loss = loss_and_grads<double>(s, E, W1, b1, w2, b2, windows, corrupt, nullptr) / B;
  return ORACLE_OK;
}

int oracle_score_f32(int V, int d, int win, int H, int B, const float* E, const float* W1,
                     const float* b1, const float* w2, const float* b2, const int32_t* windows,
                     double* scores) {
  return score<float>(Shape{V, d, win, H, B}, E, W1, b1, w2, b2, windows, scores);
}

int oracle_score_f64(int V, int d, int win, int H, int B, const double* E, const double* W1,
                     const double* b1, const double* w2, const double* b2, const int32_t* windows,
                     double* scores) {
  return score<double>(Shape{V, d, win, H, B}, E, W1, b1, w2, b2, windows, scores);
}

/* Window gather: X[b] = concat_j E[windows[b][j]], Xc[b] = E[corrupt[b]] (plain copies). */
int oracle_gather_f32(int V, int d, int win, int B, const float* E, const int32_t* windows,
                      const int32_t* corrupt, float* X, float* Xc) {
  Shape s{V, d, win, 1, B};
  int rc = check_shape(s);
  if (rc) return rc;
  if (B > 0 && (!E || !windows || !corrupt || !X || !Xc)) return ORACLE_ENULL;
  rc = check_ids(s, windows, corrupt);
  if (rc) return rc;
  for (int b = 0; b < B; ++b) {
    for (int j = 0; j < win; ++j)
      for (int t = 0; t < d; ++t)
        X[((size_t)b * win + j) * d + t] = E[(size_t)windows[(size_t)b * win + j] * d + t];
    for (int t = 0; t < d; ++t) Xc[(size_t)b * d + t] = E[(size_t)corrupt[b] * d + t];
  }
  return ORACLE_OK;
}

/* Sorted distinct rows that one step touches: ids of the windows and the corrupt ids. */
int oracle_touched_rows(int V, int win, int B, const int32_t* windows, const int32_t* corrupt,
                        int32_t* out, int32_t cap, int32_t* count) {
  Shape s{V, 1, win, 1, B};
  int rc = check_shape(s);
  if (rc) return rc;
  if (!count || (B > 0 && (!windows || !corrupt))) return ORACLE_ENULL;
  rc = check_ids(s, windows, corrupt);
  if (rc) return rc;
  std::vector<char> seen(V, 0);
  for (long i = 0; i < (long)B * win; ++i) seen[windows[i]] = 1;
  for (int b = 0; b < B; ++b) seen[corrupt[b]] = 1;
  int32_t n = 0;
  for (int r = 0; r < V; ++r)
    if (seen[r]) {
      if (out && n < cap) out[n] = r;
      ++n;
    }
  *count = n;
  return ORACLE_OK;
}

int oracle_scatter_add_f32(int rows, int d, float* table, const int32_t* idx, const float* Y,
                           long N, double alpha) {
  return scatter_add<float>(rows, d, table, idx, Y, N, alpha);
}

int oracle_scatter_add_f64(int rows, int d, double* table, const int32_t* idx, const double* Y,
                           long N, double alpha) {
  return scatter_add<double>(rows, d, table, idx, Y, N, alpha);
}

}  // extern "C"
