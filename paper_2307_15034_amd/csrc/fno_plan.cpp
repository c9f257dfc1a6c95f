// Host side of the FNO spectral-convolution library: descriptor checks, the
// truncation index map, the greedy Tucker contraction order, plan tables
// (twiddles) cached per descriptor and device, workspace sizing, and the
// C ABI entry points that enqueue the HIP kernels.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/fno_spectral_conv.h"
#include "fno_internal.h"
#include "fno_host.h"

namespace fno {
namespace {

constexpr double kPi = 3.14159265358979323846;

inline int64_t round_up(int64_t v, int64_t m) { return (v + m - 1) / m * m; }

// --------------------------------------------------------------------------
// Descriptor checks and the truncation map T_K (Sec. 2)
// --------------------------------------------------------------------------
// Detail of the last FNO_ERR_HIP on this thread (HIP error name and step).
thread_local std::string g_last_error;

fno_status hip_fail(hipError_t e, const char* what) {
  g_last_error = std::string(hipGetErrorName(e)) + " (" + std::to_string((int)e) + ") in " + what;
  return FNO_ERR_HIP;
}

int act_of(const fno_conv_desc* d) {
  switch (d->preact) {
    case FNO_PREACT_NONE: return ACT_NONE;
    case FNO_PREACT_TANH: return ACT_TANH;
    case FNO_PREACT_HARD_CLIP: return ACT_CLIP;
    case FNO_PREACT_SIGMA_CLIP: return ACT_SIGMA;
    default: return d->precision == FNO_PREC_FP16_TANH ? ACT_TANH : ACT_NONE;
  }
}

fno_status check_desc(const fno_conv_desc* d) {
  if (!d) return FNO_ERR_INVALID_ARGUMENT;
  if (d->ndim < 1 || d->ndim > 3) return FNO_ERR_INVALID_ARGUMENT;
  if (d->precision != FNO_PREC_FP32 && d->precision != FNO_PREC_FP16_TANH)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->preact < FNO_PREACT_DEFAULT || d->preact > FNO_PREACT_SIGMA_CLIP)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->preact == FNO_PREACT_SIGMA_CLIP && !(d->clip > 0.0f && d->clip <= 3.4028235e38f))
    return FNO_ERR_INVALID_ARGUMENT;  // a positive finite number of deviations
  if (d->preact == FNO_PREACT_HARD_CLIP) {
    // a positive finite bound, one that fp16 storage can hold in fp16 mode
    const float lim = d->precision == FNO_PREC_FP16_TANH ? 65504.0f : 3.4028235e38f;
    if (!(d->clip > 0.0f && d->clip <= lim)) return FNO_ERR_INVALID_ARGUMENT;
  }
  if (d->weight_kind != FNO_WEIGHT_DENSE && d->weight_kind != FNO_WEIGHT_TUCKER &&
      d->weight_kind != FNO_WEIGHT_CP)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->path_policy != FNO_PATH_MIN_RESULT && d->path_policy != FNO_PATH_MIN_NET)
    return FNO_ERR_INVALID_ARGUMENT;
  if (d->batch < 1 || d->c_in < 1 || d->c_out < 1) return FNO_ERR_INVALID_ARGUMENT;
  const int nd = d->ndim;
  for (int j = 0; j < nd; ++j) {
    const int64_t n = d->n[j], m = d->modes[j];
    if (n < 1 || m < 1) return FNO_ERR_INVALID_ARGUMENT;
    if (j < nd - 1) {
      if (2 * m > n) return FNO_ERR_INVALID_ARGUMENT;
    } else {
      if (m > n / 2 + 1) return FNO_ERR_INVALID_ARGUMENT;
    }
  }
  if (d->weight_kind == FNO_WEIGHT_TUCKER)
    for (int j = 0; j < 2 + nd; ++j)
      if (d->rank[j] < 1) return FNO_ERR_INVALID_ARGUMENT;
  if (d->weight_kind == FNO_WEIGHT_CP && d->rank[0] < 1) return FNO_ERR_INVALID_ARGUMENT;
  // Sizes the kernels cover: extents up to 65536 per axis, index math in 64
  // bits, retained counts per plane within the register tiles.
  for (int j = 0; j < nd; ++j)
    if (d->n[j] > 65536) return FNO_ERR_UNSUPPORTED;
  if (d->batch > (1 << 30) || d->c_in > (1 << 20) || d->c_out > (1 << 20))
    return FNO_ERR_UNSUPPORTED;
  const int64_t Kb = d->modes[nd - 1];
  const int64_t Ka = nd >= 2 ? 2 * d->modes[nd - 2] : 1;
  if (Kb > 128 || Ka > 128) return FNO_ERR_UNSUPPORTED;
  if (nd == 3 && 2 * d->modes[0] > 4096) return FNO_ERR_UNSUPPORTED;
  // launch-shape limits, checked here so that a call that cannot run is
  // rejected before anything is enqueued: the 3-D leading-axis kernels put
  // batch x channels on the second grid dimension, and the plane transforms
  // count planes (batch x channels x the extents before the last two axes)
  // in 31 bits
  const int64_t cmax = d->c_in > d->c_out ? d->c_in : d->c_out;
  if (nd == 3 && d->batch * cmax > 65535) return FNO_ERR_UNSUPPORTED;
  int64_t planes = d->batch * cmax;
  for (int j = 0; j + 2 < nd; ++j) planes *= d->n[j];
  if (planes > 0x7fffffff) return FNO_ERR_UNSUPPORTED;
  return FNO_OK;
}

inline int64_t mode_k(int64_t n, int64_t m, bool last, int64_t t) {
  if (last) return t;
  return t < m ? t : n - 2 * m + t;
}

inline int64_t kextent(const fno_conv_desc* d, int j) {
  return j < d->ndim - 1 ? 2 * d->modes[j] : d->modes[j];
}

inline int64_t nspatial(const fno_conv_desc* d) {
  int64_t s = 1;
  for (int j = 0; j < d->ndim; ++j) s *= d->n[j];
  return s;
}

inline int64_t kmodes(const fno_conv_desc* d) {
  int64_t s = 1;
  for (int j = 0; j < d->ndim; ++j) s *= kextent(d, j);
  return s;
}

// --------------------------------------------------------------------------
// Greedy pairwise contraction order (Sec. 4.2)
// --------------------------------------------------------------------------
struct PStep {
  int p, q;
  std::string res;
};

using Sizes = std::map<char, int64_t>;

int64_t label_size(const std::string& s, const Sizes& sz) {
  int64_t v = 1;
  for (char c : s) v *= sz.at(c);
  return v;
}

std::string keep_indices(const std::vector<std::string>& ops, int p, int q,
                         const std::string& out) {
  std::string need = out;
  for (int r = 0; r < (int)ops.size(); ++r)
    if (r != p && r != q) need += ops[r];
  std::string res;
  for (char c : ops[p])
    if (need.find(c) != std::string::npos && res.find(c) == std::string::npos) res += c;
  for (char c : ops[q])
    if (need.find(c) != std::string::npos && res.find(c) == std::string::npos) res += c;
  return res;
}

bool share_index(const std::string& a, const std::string& b) {
  for (char c : a)
    if (b.find(c) != std::string::npos) return true;
  return false;
}

std::vector<PStep> greedy_order(std::vector<std::string> ops, const Sizes& sz,
                                const std::string& out, int policy) {
  std::vector<PStep> steps;
  while (ops.size() > 1) {
    if (ops.size() == 2) {
      steps.push_back({0, 1, out});
      break;
    }
    const int n = (int)ops.size();
    bool any_share = false;
    for (int p = 0; p < n && !any_share; ++p)
      for (int q = p + 1; q < n; ++q)
        if (share_index(ops[p], ops[q])) {
          any_share = true;
          break;
        }
    bool have = false;
    int64_t best = 0;
    PStep pick{0, 1, ""};
    for (int p = 0; p < n; ++p)
      for (int q = p + 1; q < n; ++q) {
        if (any_share && !share_index(ops[p], ops[q])) continue;
        std::string res = keep_indices(ops, p, q, out);
        int64_t cost = label_size(res, sz);
        if (policy == FNO_PATH_MIN_NET) cost -= label_size(ops[p], sz) + label_size(ops[q], sz);
        if (!have || cost < best) {
          have = true;
          best = cost;
          pick = {p, q, res};
        }
      }
    steps.push_back(pick);
    std::vector<std::string> next;
    for (int r = 0; r < n; ++r)
      if (r != pick.p && r != pick.q) next.push_back(ops[r]);
    next.push_back(pick.res);
    ops.swap(next);
  }
  return steps;
}

// Memory order of the intermediates of a path (the greedy rule fixes which
// indices a result keeps, not their order): the indices of the larger input
// keep that input's order, innermost last, and the others go outermost.
// Consecutive result elements then step through the larger input
// contiguously.  The last step keeps the output's order.
std::vector<PStep> memory_order(std::vector<PStep> path, std::vector<std::string> ops,
                                const Sizes& sz) {
  for (size_t st = 0; st < path.size(); ++st) {
    PStep& ps = path[st];
    if (st + 1 < path.size()) {
      const std::string& big =
          label_size(ops[ps.p], sz) >= label_size(ops[ps.q], sz) ? ops[ps.p] : ops[ps.q];
      std::string outer, inner;
      for (char c : ps.res)
        if (big.find(c) == std::string::npos) outer += c;
      for (char c : big)
        if (ps.res.find(c) != std::string::npos) inner += c;
      ps.res = outer + inner;
    }
    std::vector<std::string> next;
    for (int r = 0; r < (int)ops.size(); ++r)
      if (r != ps.p && r != ps.q) next.push_back(ops[r]);
    next.push_back(ps.res);
    ops.swap(next);
  }
  return path;
}

// Index labels: b batch, i c_in, o c_out, a r_in, e r_out, x y z spatial,
// c d f ranks of the spatial axes.
const char kSpatial[3] = {'x', 'y', 'z'};
const char kRank[3] = {'c', 'd', 'f'};

void tucker_labels(int nd, bool adjoint, std::vector<std::string>* ops, std::string* out) {
  std::string sp, rk;
  for (int j = 0; j < nd; ++j) {
    sp += kSpatial[j];
    rk += kRank[j];
  }
  ops->clear();
  ops->push_back(std::string(adjoint ? "bo" : "bi") + sp);
  ops->push_back("ae" + rk);
  ops->push_back("ia");
  ops->push_back("oe");
  for (int j = 0; j < nd; ++j) ops->push_back(std::string(1, kSpatial[j]) + kRank[j]);
  *out = std::string(adjoint ? "bi" : "bo") + sp;
}

// CP weights (Sec. 4.6): one rank index r shared by lambda and every factor.
//   Xhat(b i x..) lambda(r) u_in(i r) u_out(o r) u_j(x_j r) -> (b o x..)
void cp_labels(int nd, bool adjoint, std::vector<std::string>* ops, std::string* out) {
  std::string sp;
  for (int j = 0; j < nd; ++j) sp += kSpatial[j];
  ops->clear();
  ops->push_back(std::string(adjoint ? "bo" : "bi") + sp);
  ops->push_back("r");
  ops->push_back("ir");
  ops->push_back("or");
  for (int j = 0; j < nd; ++j) ops->push_back(std::string(1, kSpatial[j]) + "r");
  *out = std::string(adjoint ? "bi" : "bo") + sp;
}

Sizes cp_sizes(const fno_conv_desc* d) {
  Sizes s;
  s['b'] = d->batch;
  s['i'] = d->c_in;
  s['o'] = d->c_out;
  s['r'] = d->rank[0];
  for (int j = 0; j < d->ndim; ++j) s[kSpatial[j]] = kextent(d, j);
  return s;
}

Sizes tucker_sizes(const fno_conv_desc* d) {
  Sizes s;
  s['b'] = d->batch;
  s['i'] = d->c_in;
  s['o'] = d->c_out;
  s['a'] = d->rank[0];
  s['e'] = d->rank[1];
  for (int j = 0; j < d->ndim; ++j) {
    s[kSpatial[j]] = kextent(d, j);
    s[kRank[j]] = d->rank[2 + j];
  }
  return s;
}

inline bool factorized(const fno_conv_desc* d) {
  return d->weight_kind == FNO_WEIGHT_TUCKER || d->weight_kind == FNO_WEIGHT_CP;
}

// Labels and sizes of the factorised contraction (Tucker or CP).
void weight_labels(const fno_conv_desc* d, bool adjoint, std::vector<std::string>* ops,
                   std::string* out) {
  if (d->weight_kind == FNO_WEIGHT_CP) cp_labels(d->ndim, adjoint, ops, out);
  else tucker_labels(d->ndim, adjoint, ops, out);
}

Sizes weight_sizes(const fno_conv_desc* d) {
  return d->weight_kind == FNO_WEIGHT_CP ? cp_sizes(d) : tucker_sizes(d);
}

int32_t label_bit(char c) {
  switch (c) {
    case 'r': return 11;
    case 'b': return 0;
    case 'i': return 1;
    case 'o': return 2;
    case 'a': return 3;
    case 'e': return 4;
    case 'x': return 5;
    case 'y': return 6;
    case 'z': return 7;
    case 'c': return 8;
    case 'd': return 9;
    case 'f': return 10;
  }
  return 31;
}

// --------------------------------------------------------------------------
// Plans: geometry and device tables
// --------------------------------------------------------------------------
struct Geo {
  int nd;
  int elem;          // ELEM_F16 / ELEM_F32
  int es;            // element bytes
  int act;           // pre-activation: ACT_NONE / ACT_TANH / ACT_CLIP / ACT_SIGMA
  float clip;        // bound of ACT_CLIP; deviations of ACT_SIGMA
  int64_t B, Cin, Cout;
  int64_t N;         // prod n
  int64_t K;         // prod K_j
  // plane transform (last two axes)
  int Na, Nb, Ka, Kb;
  int Kbp, nct;
  int Nbp, Kap16;
  int R_f, Nap_f;    // r2c chunking
  int Kap, R_i, Nap_i, Nb64;  // c2r
  int NaC;           // Na padded to 32 (chained forward tables)
  // leading 3-D axis
  int N1, K1, Lin_f, Linp_f, Lout16_f, Linp_i, Lout16_i;
  // radix-2 wide-plane transforms (fp16 planes with both extents multiples
  // of 256): column tiles per class, leading-axis tiles per class, and the
  // leading-axis slots per class padded to 32
  int w2, w2_nctc, w2_nta, w2_kah;
};

struct DevTables {
  void* base = nullptr;
  size_t bytes = 0;
  const void *zeros, *twA, *cB, *sB, *cI, *sI, *twI;
  const void *twAc, *cBc, *sBc, *twIc, *cIc, *sIc;
  const void *lutAct, *lutGrad;
  int actSat = 0, gradSat = 0;  // first codes of the saturated tails (fp16 plans)
  const void *eFr, *eFi, *eIr, *eIi;
  const void *twA2, *cB2, *sB2, *cI2, *sI2, *twI2;  // radix-2 wide-plane tables
};

struct Plan {
  Geo g;
  DevTables t;
  int num_cu = 256;
  std::vector<PStep> path_fwd, path_adj;
  std::vector<std::string> labels_fwd, labels_adj;
  std::string out_fwd, out_adj;
  int device = 0;
  // early requests in the narrow wide-plane forward (see host_plan)
  bool r2c_early = true;
  Plan() = default;
  Plan(const Plan&) = delete;
  Plan& operator=(const Plan&) = delete;
  // the device tables go with the last reference (the cache's, or that of a
  // call still running on another thread when the cache is released)
  ~Plan() {
    if (!t.base) return;
    int cur = 0;
    (void)hipGetDevice(&cur);
    (void)hipSetDevice(device);
    (void)hipFree(t.base);
    (void)hipSetDevice(cur);
  }
};

Geo make_geo(const fno_conv_desc* d) {
  Geo g{};
  g.nd = d->ndim;
  g.elem = d->precision == FNO_PREC_FP16_TANH ? ELEM_F16 : ELEM_F32;
  g.es = g.elem == ELEM_F16 ? 2 : 4;
  g.act = act_of(d);
  g.clip = g.act == ACT_CLIP || g.act == ACT_SIGMA ? d->clip : 0.0f;
  g.B = d->batch;
  g.Cin = d->c_in;
  g.Cout = d->c_out;
  g.N = nspatial(d);
  g.K = kmodes(d);
  const int nd = d->ndim;
  g.Nb = (int)d->n[nd - 1];
  g.Kb = (int)d->modes[nd - 1];
  if (nd >= 2) {
    g.Na = (int)d->n[nd - 2];
    g.Ka = (int)(2 * d->modes[nd - 2]);
  } else {
    g.Na = 1;
    g.Ka = 1;
  }
  int kb16 = (int)round_up(g.Kb, 16);
  int kbp = 16;
  while (kbp < kb16) kbp *= 2;
  g.Kbp = kbp;
  g.nct = 2 * kbp / 16;
  g.Nbp = (int)round_up(g.Nb, 32);
  g.Kap16 = (int)round_up(g.Ka, 16);
  // r2c row chunk: step-A result of one chunk stays within ~32 KiB of LDS
  int rmax = (int)(32768 / (2 * g.Kbp * g.es)) / 32 * 32;
  rmax = std::max(32, rmax);
  g.R_f = (int)std::min<int64_t>(round_up(g.Na, 32), rmax);
  g.Nap_f = (int)round_up(g.Na, g.R_f);
  // c2r
  g.Kap = (int)round_up(g.Ka, 32);
  int rmaxi = (int)(32768 / (2 * g.Kbp * g.es)) / 16 * 16;
  rmaxi = std::max(16, rmaxi);
  g.R_i = (int)std::min<int64_t>(round_up(g.Na, 16), rmaxi);
  g.Nap_i = (int)round_up(g.Na, g.R_i);
  g.Nb64 = (int)round_up(g.Nb, 64);
  g.NaC = (int)round_up(g.Na, 32);
  if (nd == 3) {
    g.N1 = (int)d->n[0];
    g.K1 = (int)(2 * d->modes[0]);
    g.Linp_f = (int)round_up(g.N1, 32);
    g.Lout16_f = (int)round_up(g.K1, 16);
    g.Linp_i = (int)round_up(g.K1, 32);
    g.Lout16_i = (int)round_up(g.N1, 16);
  }
  g.w2 = 0;
  if (g.elem == ELEM_F16 && nd == 2 && g.Na % 256 == 0 && g.Nb % 256 == 0 && g.Kb <= 64 &&
      g.Kb % 4 == 0 && g.Ka <= 128 && g.Ka * g.Kb <= 8192 &&
      (int64_t)g.Na * g.Nb * 2 < ((int64_t)1 << 30)) {
    const int kbe = (g.Kb + 1) / 2, m = g.Ka / 2;
    const int nta = (m + 15) / 16;
    g.w2 = 1;
    g.w2_nctc = kbe <= 16 ? 2 : 4;
    g.w2_nta = nta <= 1 ? 1 : nta <= 2 ? 2 : 4;
    g.w2_kah = (int)round_up(m, 32);
  }
  return g;
}

// cos/sin of 2 pi (k n mod N) / N with the phase reduced exactly in integers.
inline void twiddle(int64_t k, int64_t n, int64_t N, double* c, double* s) {
  const int64_t r = ((k % N) * (n % N)) % N;
  const double ph = 2.0 * kPi * (double)r / (double)N;
  *c = std::cos(ph);
  *s = std::sin(ph);
}

template <typename T>
void fill_tables(const fno_conv_desc* d, const Geo& g, std::vector<T>& buf,
                 std::vector<size_t>& off) {
  auto alloc = [&](size_t n) {
    size_t o = round_up((int64_t)buf.size(), 64);
    buf.resize(o + n, (T)0.0f);
    off.push_back(o);
    return o;
  };
  alloc(256 / sizeof(T));  // zero block: loads of out-of-range lanes point here
  const int nd = g.nd;
  const int64_t ma = nd >= 2 ? d->modes[nd - 2] : 1;
  auto ka_of = [&](int t) -> int64_t {
    return nd >= 2 ? mode_k(g.Na, ma, false, t) : 0;
  };
  // twA [2 Kbp][Nbp]
  size_t o = alloc((size_t)2 * g.Kbp * g.Nbp);
  for (int t = 0; t < g.Kb; ++t)
    for (int n = 0; n < g.Nb; ++n) {
      double c, s;
      twiddle(t, n, g.Nb, &c, &s);
      buf[o + (size_t)t * g.Nbp + n] = (T)c;
      buf[o + (size_t)(g.Kbp + t) * g.Nbp + n] = (T)(-s);
    }
  // cB, sB [Kap16][Nap_f]
  size_t oc = alloc((size_t)g.Kap16 * g.Nap_f);
  size_t os = alloc((size_t)g.Kap16 * g.Nap_f);
  for (int t = 0; t < g.Ka; ++t)
    for (int n = 0; n < g.Na; ++n) {
      double c, s;
      twiddle(ka_of(t), n, g.Na, &c, &s);
      buf[oc + (size_t)t * g.Nap_f + n] = (T)c;
      buf[os + (size_t)t * g.Nap_f + n] = (T)s;
    }
  // cI, sI [Nap_i][Kap]
  size_t oci = alloc((size_t)g.Nap_i * g.Kap);
  size_t osi = alloc((size_t)g.Nap_i * g.Kap);
  for (int n = 0; n < g.Na; ++n)
    for (int t = 0; t < g.Ka; ++t) {
      double c, s;
      twiddle(ka_of(t), n, g.Na, &c, &s);
      buf[oci + (size_t)n * g.Kap + t] = (T)c;
      buf[osi + (size_t)n * g.Kap + t] = (T)s;
    }
  // twI [Nb64][2 Kbp]
  size_t oti = alloc((size_t)g.Nb64 * 2 * g.Kbp);
  for (int n = 0; n < g.Nb; ++n)
    for (int t = 0; t < g.Kb; ++t) {
      double c, s;
      twiddle(t, n, g.Nb, &c, &s);
      buf[oti + (size_t)n * 2 * g.Kbp + t] = (T)c;
      buf[oti + (size_t)n * 2 * g.Kbp + g.Kbp + t] = (T)(-s);
    }
  // Permuted copies for the chained kernels (whose MFMA results feed the
  // next MFMA directly).  twAc [2 Kbp][Nbp]: row 16 ct + r holds part
  // ct / ntb (cos, then -sin) of t = ntb r + ct % ntb.
  const int ntb = g.Kbp / 16;
  size_t oac = alloc((size_t)2 * g.Kbp * g.Nbp);
  for (int ct = 0; ct < 2 * ntb; ++ct)
    for (int r = 0; r < 16; ++r) {
      const int part = ct / ntb, t = ntb * r + ct % ntb;
      if (t >= g.Kb) continue;
      for (int n = 0; n < g.Nb; ++n) {
        double c, s;
        twiddle(t, n, g.Nb, &c, &s);
        buf[oac + (size_t)(ct * 16 + r) * g.Nbp + n] = (T)(part == 0 ? c : -s);
      }
    }
  // cBc, sBc [Kap16][NaC]: column 32 j + 8 q + e holds row
  // n = 32 j + 4 q + e (e < 4) or 32 j + 16 + 4 q + (e - 4) (e >= 4)
  size_t obc = alloc((size_t)g.Kap16 * g.NaC);
  size_t obs = alloc((size_t)g.Kap16 * g.NaC);
  for (int t = 0; t < g.Ka; ++t)
    for (int col = 0; col < g.NaC; ++col) {
      const int j = col / 32, q = (col % 32) / 8, e = col % 8;
      const int n = 32 * j + (e < 4 ? 4 * q + e : 16 + 4 * q + (e - 4));
      if (n >= g.Na) continue;
      double c, s;
      twiddle(ka_of(t), n, g.Na, &c, &s);
      buf[obc + (size_t)t * g.NaC + col] = (T)c;
      buf[obs + (size_t)t * g.NaC + col] = (T)s;
    }
  // twIc [Nb64][2 Kbp]: row 16 T + R holds n = 64 (T/4) + 16 (R/4) + 4 (T%4)
  // + R%4; column 32 ks + 8 q + e holds pair 2 ks + e/4 (pairs: Re tiles
  // 0..ntb-1, then Im tiles) at t = 16 tile + 4 q + e%4; Re: cos, Im: -sin
  size_t oic = alloc((size_t)g.Nb64 * 2 * g.Kbp);
  for (int row = 0; row < g.Nb64; ++row) {
    const int tile16 = row / 16, R = row % 16;
    const int n = 64 * (tile16 / 4) + 16 * (R / 4) + 4 * (tile16 % 4) + R % 4;
    if (n >= g.Nb) continue;
    for (int col = 0; col < 2 * g.Kbp; ++col) {
      const int ks = col / 32, q = (col % 32) / 8, e = col % 8;
      const int pair = 2 * ks + e / 4;
      const int part = pair / ntb, tile = pair % ntb;
      const int t = 16 * tile + 4 * q + e % 4;
      if (t >= g.Kb) continue;
      double c, s;
      twiddle(t, n, g.Nb, &c, &s);
      buf[oic + (size_t)row * 2 * g.Kbp + col] = (T)(part == 0 ? c : -s);
    }
  }
  // cIc, sIc [Nap_i][Kap]: cI, sI with column 32 ks + 8 q + e holding
  // t = 32 ks + 4 q + e (e < 4) or 32 ks + 16 + 4 q + (e - 4)
  size_t oicc = alloc((size_t)g.Nap_i * g.Kap);
  size_t oics = alloc((size_t)g.Nap_i * g.Kap);
  for (int n = 0; n < g.Na; ++n)
    for (int col = 0; col < g.Kap; ++col) {
      const int ks = col / 32, q = (col % 32) / 8, e = col % 8;
      const int t = 32 * ks + (e < 4 ? 4 * q + e : 16 + 4 * q + (e - 4));
      if (t >= g.Ka) continue;
      double c, s;
      twiddle(ka_of(t), n, g.Na, &c, &s);
      buf[oicc + (size_t)n * g.Kap + col] = (T)c;
      buf[oics + (size_t)n * g.Kap + col] = (T)s;
    }
  // Lookup tables over the non-negative fp16 codes 0..0x7fff: the
  // pre-activation f and its derivative f' of the fp16 value, each rounded
  // once to the storage type.  tanh: f = tanh, f' = sech^2 = 1 - tanh^2
  // (+inf gives 1 and 0); hard clip: f = min(x, clip), f' = 1 up to clip and
  // 0 beyond.  NaN codes give NaN in both.  f is odd and f' even, so the
  // kernels look up |x| and restore the sign of f.
  size_t olt = alloc(32768);
  size_t ols = alloc(32768);
  const double cb = (double)g.clip;
  for (int code = 0; code < 32768; ++code) {
    const uint16_t bits = (uint16_t)code;
    _Float16 h;
    std::memcpy(&h, &bits, 2);
    const double xv = (double)h;
    double f, fp;
    if (std::isnan(xv)) {
      f = fp = xv;
    } else if (g.act == ACT_CLIP) {
      f = xv > cb ? cb : xv;
      fp = xv <= cb ? 1.0 : 0.0;
    } else {
      const double ch = std::cosh(xv);
      f = std::tanh(xv);
      fp = 1.0 / (ch * ch);
    }
    buf[olt + code] = (T)f;
    buf[ols + code] = (T)fp;
  }
  (void)o;
  (void)oc;
  (void)os;
  (void)oci;
  (void)osi;
  (void)oti;
  if (g.w2) {
    // radix-2 wide-plane tables (even and odd slots of each axis as classes)
    const int kbpc = g.w2_nctc * 8, nh = g.Nb / 2, nha = g.Na / 2, m = g.Ka / 2;
    const int nta16 = g.w2_nta * 16, kah = g.w2_kah;
    // twA2 [4 kbpc][nh]: row cls 2 kbpc + c: cos, + kbpc: -sin of 2 pi k n / Nb
    size_t a2 = alloc((size_t)4 * kbpc * nh);
    // twI2 [nh][4 kbpc]: the same values, transposed
    size_t i2 = alloc((size_t)nh * 4 * kbpc);
    for (int cls = 0; cls < 2; ++cls)
      for (int c = 0; c < kbpc; ++c) {
        const int k = 2 * c + cls;
        if (k >= g.Kb) continue;
        for (int n = 0; n < nh; ++n) {
          double cv, sv;
          twiddle(k, n, g.Nb, &cv, &sv);
          buf[a2 + (size_t)(cls * 2 * kbpc + c) * nh + n] = (T)cv;
          buf[a2 + (size_t)(cls * 2 * kbpc + kbpc + c) * nh + n] = (T)(-sv);
          buf[i2 + (size_t)n * 4 * kbpc + cls * 2 * kbpc + c] = (T)cv;
          buf[i2 + (size_t)n * 4 * kbpc + cls * 2 * kbpc + kbpc + c] = (T)(-sv);
        }
      }
    // cB2, sB2 [2][nta16][nha]; cI2, sI2 [2][nha][kah]: slot t_a = 2 t + cls
    size_t cb2 = alloc((size_t)2 * nta16 * nha), sb2 = alloc((size_t)2 * nta16 * nha);
    size_t ci2 = alloc((size_t)2 * nha * kah), si2 = alloc((size_t)2 * nha * kah);
    for (int cls = 0; cls < 2; ++cls)
      for (int t = 0; t < m; ++t) {
        const int64_t ka = ka_of(2 * t + cls);
        for (int r = 0; r < nha; ++r) {
          double cv, sv;
          twiddle(ka, r, g.Na, &cv, &sv);
          buf[cb2 + ((size_t)cls * nta16 + t) * nha + r] = (T)cv;
          buf[sb2 + ((size_t)cls * nta16 + t) * nha + r] = (T)sv;
          buf[ci2 + ((size_t)cls * nha + r) * kah + t] = (T)cv;
          buf[si2 + ((size_t)cls * nha + r) * kah + t] = (T)sv;
        }
      }
  }
  if (nd == 3) {
    const int64_t m1 = d->modes[0];
    // forward E[t][l] = exp(-2 pi i k1(t) l / N1): [Lout16_f][Linp_f]
    size_t er = alloc((size_t)g.Lout16_f * g.Linp_f);
    size_t ei = alloc((size_t)g.Lout16_f * g.Linp_f);
    for (int t = 0; t < g.K1; ++t)
      for (int l = 0; l < g.N1; ++l) {
        double c, s;
        twiddle(mode_k(g.N1, m1, false, t), l, g.N1, &c, &s);
        buf[er + (size_t)t * g.Linp_f + l] = (T)c;
        buf[ei + (size_t)t * g.Linp_f + l] = (T)(-s);
      }
    // inverse E[n][t] = exp(+2 pi i k1(t) n / N1): [Lout16_i][Linp_i]
    size_t ir = alloc((size_t)g.Lout16_i * g.Linp_i);
    size_t ii = alloc((size_t)g.Lout16_i * g.Linp_i);
    for (int n = 0; n < g.N1; ++n)
      for (int t = 0; t < g.K1; ++t) {
        double c, s;
        twiddle(mode_k(g.N1, m1, false, t), n, g.N1, &c, &s);
        buf[ir + (size_t)n * g.Linp_i + t] = (T)c;
        buf[ii + (size_t)n * g.Linp_i + t] = (T)s;
      }
  }
}

struct PlanKey {
  std::array<int64_t, 24> v;
  bool operator<(const PlanKey& o) const { return v < o.v; }
};

PlanKey key_of(const fno_conv_desc* d, int device) {
  PlanKey k;
  k.v.fill(0);
  k.v[0] = device;
  k.v[1] = d->ndim;
  k.v[2] = d->precision;
  k.v[3] = d->weight_kind;
  k.v[4] = d->path_policy;
  k.v[5] = d->batch;
  k.v[6] = d->c_in;
  k.v[7] = d->c_out;
  for (int j = 0; j < d->ndim; ++j) {
    k.v[8 + j] = d->n[j];
    k.v[11 + j] = d->modes[j];
  }
  if (d->weight_kind == FNO_WEIGHT_TUCKER)
    for (int j = 0; j < 2 + d->ndim; ++j) k.v[14 + j] = d->rank[j];
  if (d->weight_kind == FNO_WEIGHT_CP) k.v[14] = d->rank[0];
  const int act = act_of(d);
  k.v[19] = act;
  if (act == ACT_CLIP || act == ACT_SIGMA) {
    uint32_t bits;
    std::memcpy(&bits, &d->clip, 4);
    k.v[20] = bits;
  }
  return k;
}

std::mutex g_mutex;
std::map<PlanKey, std::shared_ptr<Plan>> g_plans;

fno_status build_tables(const fno_conv_desc* d, Plan* pl) {
  std::vector<size_t> off;
  size_t bytes = 0;
  std::vector<_Float16> b16;
  std::vector<float> b32;
  if (pl->g.elem == ELEM_F16) {
    fill_tables<_Float16>(d, pl->g, b16, off);
    bytes = b16.size() * 2;
    // the tanh and sech^2 tables are constant from some code up to +inf
    // (0x7c00): the wide-plane kernels keep only the codes below in LDS
    auto sat_of = [&](size_t o) {
      uint16_t top, v;
      std::memcpy(&top, &b16[o + 0x7c00], 2);
      int c = 0x7c00;
      for (; c > 0; --c) {
        std::memcpy(&v, &b16[o + c - 1], 2);
        if (v != top) break;
      }
      return c;
    };
    pl->t.actSat = sat_of(off[13]);
    pl->t.gradSat = sat_of(off[14]);
  } else {
    fill_tables<float>(d, pl->g, b32, off);
    bytes = b32.size() * 4;
  }
  void* dev = nullptr;
  hipError_t e = hipMalloc(&dev, std::max<size_t>(bytes, 256));
  if (e != hipSuccess) return hip_fail(e, "hipMalloc (plan tables)");
  const void* src = pl->g.elem == ELEM_F16 ? (const void*)b16.data() : (const void*)b32.data();
  e = hipMemcpy(dev, src, bytes, hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(dev);
    return hip_fail(e, "hipMemcpy (plan tables)");
  }
  pl->t.base = dev;
  pl->t.bytes = bytes;
  auto at = [&](int i) -> const void* {
    return (const void*)((const char*)dev + off[i] * pl->g.es);
  };
  pl->t.zeros = at(0);
  pl->t.twA = at(1);
  pl->t.cB = at(2);
  pl->t.sB = at(3);
  pl->t.cI = at(4);
  pl->t.sI = at(5);
  pl->t.twI = at(6);
  pl->t.twAc = at(7);
  pl->t.cBc = at(8);
  pl->t.sBc = at(9);
  pl->t.twIc = at(10);
  pl->t.cIc = at(11);
  pl->t.sIc = at(12);
  pl->t.lutAct = at(13);
  pl->t.lutGrad = at(14);
  if (pl->g.w2) {  // allocated after the lookup tables (2-D plans only)
    pl->t.twA2 = at(15);
    pl->t.twI2 = at(16);
    pl->t.cB2 = at(17);
    pl->t.sB2 = at(18);
    pl->t.cI2 = at(19);
    pl->t.sI2 = at(20);
  }
  if (pl->g.nd == 3) {
    pl->t.eFr = at(15);
    pl->t.eFi = at(16);
    pl->t.eIr = at(17);
    pl->t.eIi = at(18);
  }
  return FNO_OK;
}

// Geometry and Tucker paths: host-only, no device calls.
void host_plan(const fno_conv_desc* d, Plan* pl) {
  pl->g = make_geo(d);
  // The early-request forward holds 32 more registers per wave.  The
  // MIN_RESULT factorised paths run their longest weights-only products on a
  // side stream beside the forward transform, and those slow down more
  // (fewer registers left on each SIMD) than the transform gains; with
  // MIN_NET and dense weights the early requests are faster.
  pl->r2c_early = !(factorized(d) && d->path_policy == FNO_PATH_MIN_RESULT);
  if (factorized(d)) {
    Sizes sz = weight_sizes(d);
    weight_labels(d, false, &pl->labels_fwd, &pl->out_fwd);
    weight_labels(d, true, &pl->labels_adj, &pl->out_adj);
    pl->path_fwd = memory_order(
        greedy_order(pl->labels_fwd, sz, pl->out_fwd, d->path_policy), pl->labels_fwd, sz);
    pl->path_adj = memory_order(
        greedy_order(pl->labels_adj, sz, pl->out_adj, d->path_policy), pl->labels_adj, sz);
  }
}

// The plan of a descriptor on the current device, built on first use.  The
// caller holds a reference for the duration of its call, so a concurrent
// fno_release_caches cannot free the tables under it.
fno_status get_plan(const fno_conv_desc* d, std::shared_ptr<Plan>* out, bool build = true) {
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  int dev = 0;
  const hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  PlanKey key = key_of(d, dev);
  std::lock_guard<std::mutex> lock(g_mutex);
  auto it = g_plans.find(key);
  if (it != g_plans.end()) {
    *out = it->second;
    return FNO_OK;
  }
  if (!build) {
    g_last_error = "no plan for this descriptor on this device: make one ordinary call first";
    return FNO_ERR_INVALID_ARGUMENT;
  }
  std::shared_ptr<Plan> pl = std::make_shared<Plan>();
  host_plan(d, pl.get());
  pl->device = dev;
  int ncu = 0;
  if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess &&
      ncu > 0)
    pl->num_cu = ncu;
  st = build_tables(d, pl.get());
  if (st != FNO_OK) return st;
  *out = pl;
  g_plans[key] = std::move(pl);
  return FNO_OK;
}

// --------------------------------------------------------------------------
// Workspace layout
// --------------------------------------------------------------------------
struct WsLayout {
  size_t total = 0;
  size_t add(size_t bytes) {
    size_t o = total;
    total += (size_t)round_up((int64_t)std::max<size_t>(bytes, 1), 256);
    return o;
  }
};

size_t spec_bytes(const Geo& g, int64_t C) { return (size_t)g.B * C * g.K * 2 * g.es; }

size_t inter3d_bytes(const Geo& g, int64_t C) {
  if (g.nd != 3) return 0;
  return (size_t)g.B * C * g.N1 * g.Ka * g.Kb * 2 * g.es;
}

struct TuckerWs {
  std::vector<size_t> step_off;  // one fp32 complex buffer per intermediate
  size_t total = 0;
};

// Tucker intermediates of a path (all but the last step, which writes the
// output spectrum).
size_t tucker_path_bytes(const fno_conv_desc* d, const std::vector<PStep>& path) {
  Sizes sz = weight_sizes(d);
  size_t t = kPairPartBytes;  // split-K partial sums
  for (size_t s = 0; s + 1 < path.size(); ++s)
    t += (size_t)round_up(label_size(path[s].res, sz) * 8, 256);
  return t;
}

size_t tucker_wgrad_bytes(const fno_conv_desc* d, const Plan* pl);
size_t cp_wgrad_bytes(const fno_conv_desc* d, const Plan* pl);

size_t ws_bytes(const fno_conv_desc* d, const Plan* pl, fno_op op, bool caches);

// The workspace without the clip bounds of the statistics-based
// pre-activation (a multiple of 256 bytes; the bounds follow it).
size_t ws_core(const fno_conv_desc* d, const Plan* pl, fno_op op, bool caches) {
  const Geo& g = pl->g;
  WsLayout w;
  const bool tucker = factorized(d);
  if (op == FNO_OP_FWD) {
    w.add(spec_bytes(g, g.Cin));
    w.add(spec_bytes(g, g.Cout));
    w.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
    if (tucker) w.add(tucker_path_bytes(d, pl->path_fwd));
  } else if (op == FNO_OP_BWD_DATA) {
    w.add(spec_bytes(g, g.Cout));
    w.add(spec_bytes(g, g.Cin));
    w.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
    if (tucker) w.add(tucker_path_bytes(d, pl->path_adj));
  } else if (op == FNO_OP_BWD_WEIGHT) {
    if (!caches) {
      w.add(spec_bytes(g, g.Cin));
      w.add(spec_bytes(g, g.Cout));
      w.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
    }
    if (tucker)
      w.add(d->weight_kind == FNO_WEIGHT_CP ? cp_wgrad_bytes(d, pl) : tucker_wgrad_bytes(d, pl));
  } else {  // FNO_OP_BWD: gradient spectrum, input spectrum (no cache), then
            // the data part's workspace and (Tucker) the weight part's
    w.add(spec_bytes(g, g.Cout));
    if (!caches) w.add(spec_bytes(g, g.Cin));
    w.add(ws_bytes(d, pl, FNO_OP_BWD_DATA, true));
    if (tucker) w.add(ws_bytes(d, pl, FNO_OP_BWD_WEIGHT, true));
  }
  return std::max<size_t>((size_t)round_up((int64_t)w.total, 256), 256);
}

// Clip bounds (lo, hi in double) of every (batch, input channel) plane: held
// by the forward, data-gradient and cache-less weight-gradient workspaces
// (the combined backward uses its data part's).
size_t bounds_bytes(const Plan* pl, fno_op op, bool caches) {
  const Geo& g = pl->g;
  if (g.act != ACT_SIGMA) return 0;
  if (op == FNO_OP_BWD || (op == FNO_OP_BWD_WEIGHT && caches)) return 0;
  return (size_t)round_up(g.B * g.Cin * 16, 256);
}

size_t ws_bytes(const fno_conv_desc* d, const Plan* pl, fno_op op, bool caches) {
  return ws_core(d, pl, op, caches) + bounds_bytes(pl, op, caches);
}

// Computes the clip bounds of x into `bounds` when the plan's pre-activation
// is the statistics-based clip (nothing otherwise).
fno_status run_sigma_stats(const Plan* pl, const void* x, double* bounds, hipStream_t s);

// --------------------------------------------------------------------------
// Kernel sequences
// --------------------------------------------------------------------------
inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

#define FNO_HIP(call)                          \
  do {                                         \
    const hipError_t fno_e_ = (call);          \
    if (fno_e_ != hipSuccess) return hip_fail(fno_e_, #call); \
  } while (0)

// --------------------------------------------------------------------------
// Optional per-kernel event timing
// --------------------------------------------------------------------------
struct ProfEntry {
  std::string name;
  int64_t launches = 0;
  double total_ms = 0.0;
};
struct Pending {
  int slot;
  hipEvent_t a, b;
};
std::mutex g_prof_mutex;
bool g_prof_on = false;
std::vector<ProfEntry> g_prof;
std::vector<Pending> g_pending;

int prof_slot(const char* name) {
  for (size_t i = 0; i < g_prof.size(); ++i)
    if (g_prof[i].name == name) return (int)i;
  g_prof.push_back(ProfEntry{name, 0, 0.0});
  return (int)g_prof.size() - 1;
}

// Runs `launch` bracketed by events when profiling is on.
// set while the calling thread runs an allocation-free entry point (no
// events are created for it)
thread_local bool g_no_alloc_call = false;

template <typename F>
hipError_t timed(const char* name, hipStream_t s, F launch) {
  bool on;
  {
    std::lock_guard<std::mutex> lk(g_prof_mutex);
    on = g_prof_on;
  }
  if (!on || g_no_alloc_call) return launch();
  hipEvent_t a = nullptr, b = nullptr;
  if (hipEventCreate(&a) != hipSuccess) return hipErrorOutOfMemory;
  if (hipEventCreate(&b) != hipSuccess) {
    (void)hipEventDestroy(a);
    return hipErrorOutOfMemory;
  }
  (void)hipEventRecord(a, s);
  hipError_t e = launch();
  (void)hipEventRecord(b, s);
  std::lock_guard<std::mutex> lk(g_prof_mutex);
  g_pending.push_back(Pending{prof_slot(name), a, b});
  return e;
}

void prof_drain() {
  for (Pending& p : g_pending) {
    (void)hipEventSynchronize(p.b);
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      g_prof[p.slot].launches += 1;
      g_prof[p.slot].total_ms += ms;
    }
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  g_pending.clear();
}

// Forward truncated transform of planes -> spectrum [B][C][K...].
// scale_mode 0: 1/N normalisation (input spectrum), 1: 1/sqrt(N) (gradient).
// pre: apply the plan's pre-activation (if it has one) to the input.
fno_status run_sigma_stats(const Plan* pl, const void* x, double* bounds, hipStream_t s) {
  const Geo& g = pl->g;
  if (g.act != ACT_SIGMA) return FNO_OK;
  FNO_HIP(timed("sigma_stats", s, [&] {
    return launch_sigma_stats(g.elem, x, g.B * g.Cin, g.N, (double)g.clip, bounds, s);
  }));
  return FNO_OK;
}

// bounds: the clip bounds of the statistics-based pre-activation (read when
// it is applied to the input).
fno_status run_r2c(const Plan* pl, const void* in, void* spec, void* inter, int64_t C,
                   int pre, int scale_mode, hipStream_t s, const double* bounds = nullptr) {
  const Geo& g = pl->g;
  R2CArgs a{};
  a.zeros = pl->t.zeros;
  a.in = in;
  a.out = g.nd == 3 ? inter : spec;
  a.twA = pl->t.twA;
  a.cB = pl->t.cB;
  a.sB = pl->t.sB;
  a.planes = g.B * C * (g.nd == 3 ? g.N1 : 1);
  a.Na = g.Na;
  a.Nb = g.Nb;
  a.Ka = g.Ka;
  a.Kb = g.Kb;
  a.Kbp = g.Kbp;
  a.Nbp = g.Nbp;
  a.Nap = g.Nap_f;
  a.Kap16 = g.Kap16;
  a.R = g.R_f;
  if (scale_mode == 0) {
    a.scaleA = (float)(1.0 / g.Nb);
    a.scaleB = (float)(1.0 / g.Na);
  } else {
    a.scaleA = (float)(1.0 / std::sqrt((double)g.Nb));
    a.scaleB = (float)(1.0 / std::sqrt((double)g.Na));
  }
  a.do_tanh = pre && g.act != ACT_NONE;
  a.act = a.do_tanh ? g.act : ACT_NONE;
  a.clip = g.clip;
  const bool do_tanh = a.do_tanh;
  const char* kname = !do_tanh                ? "r2c_plane"
                      : g.act == ACT_TANH      ? "r2c_plane_tanh"
                      : g.act == ACT_CLIP      ? "r2c_plane_clip"
                                               : "r2c_plane_sigma";
  a.vec = (g.Nb % 8) == 0;
  // the statistics-based clip has per-plane bounds, no table: the
  // table-free kernel only
  const bool sigma = do_tanh && g.act == ACT_SIGMA;
  if (sigma) {
    if (!bounds) return FNO_ERR_INTERNAL;
    a.bounds = bounds;
    a.bgroup = g.nd == 3 ? g.N1 : 1;
  }
  a.twAc = pl->t.twAc;
  a.cBc = pl->t.cBc;
  a.sBc = pl->t.sBc;
  a.NaC = g.NaC;
  a.lut = pl->t.lutAct;
  if (a.planes > 0x7fffffff || (g.nd == 3 && g.B * C > 65535)) return FNO_ERR_UNSUPPORTED;
  bool done = sigma;
  if (!done && g.elem == ELEM_F16 && a.vec && g.Kb % 4 == 0 && g.Nb <= 256 && g.Na <= 128) {
    const int nka = g.Nbp / 32, ntb = g.Kbp / 16, nta = g.Kap16 / 16;
    const size_t lds = r2c_chain_lds_bytes(nka, ntb, nta, g.NaC, do_tanh);
    const int64_t waves = (int64_t)kChainWaves;
    const int grid = (int)std::min<int64_t>((a.planes + waves - 1) / waves, (int64_t)2 * pl->num_cu);
    const size_t lut = do_tanh ? 65536 : 0;  // static LDS of the kernel
    if (lds + lut <= 160 * 1024 && grid > 0 && r2c_chain_has(nka, ntb, nta)) {
      hipError_t e = timed(kname, s, [&] {
        return launch_r2c_chain(a, nka, ntb, nta, grid, lds, s);
      });
      if (e == hipSuccess) done = true;
      else if (e != hipErrorNotSupported) return hip_fail(e, kname);
    }
  }
  if (!done && g.elem == ELEM_F16 && a.vec && g.Nb <= 256 && g.Na <= 128 && g.nct <= 8) {
    const int nka = g.Nb <= 32 ? 1 : g.Nb <= 64 ? 2 : g.Nb <= 128 ? 4 : 8;
    const int nw = g.Na <= 64 ? 4 : 8;
    const size_t lds = r2c_fast_lds_bytes(g.nct, nka, nw, g.Kap16, g.Nap_f);
    const int grid = (int)std::min<int64_t>(a.planes, (int64_t)2 * pl->num_cu);
    if (lds <= 80 * 1024) {
      hipError_t e = timed(kname, s, [&] {
        return launch_r2c_fast(a, g.nct, nka, nw, grid, lds, s);
      });
      if (e == hipSuccess) done = true;
      else if (e != hipErrorNotSupported) return hip_fail(e, kname);
    }
  }
  if (!done && g.w2) {
    // large planes, one radix-2 stage per axis: persistent eight-wave
    // work-groups, one per compute unit
    R2CArgs b = a;
    b.twA = pl->t.twA2;
    b.cB = pl->t.cB2;
    b.sB = pl->t.sB2;
    b.Kap16 = g.w2_nta * 16;
    b.lut_sat = pl->t.actSat;
    b.early = pl->r2c_early ? 1 : 0;
    const size_t lds = r2c_wide2_lds_bytes(g.w2_nctc, do_tanh, b.lut_sat);
    const int grid = (int)std::min<int64_t>(a.planes, (int64_t)pl->num_cu);
    hipError_t e = timed(kname, s, [&] { return launch_r2c_wide2(b, g.w2_nctc, grid, lds, s); });
    if (e == hipSuccess) done = true;
    else if (e != hipErrorNotSupported) return hip_fail(e, kname);
  }
  if (!done && g.elem == ELEM_F16 && g.Nb % 128 == 0 && g.Na % 256 == 0 && g.Nbp == g.Nb &&
      (g.nct == 4 || g.nct == 8) && g.Kap16 <= 128 && 128 % g.Kap16 == 0 &&
      g.Na * (int64_t)g.Nb * 2 < ((int64_t)1 << 30)) {
    // large planes: persistent eight-wave work-groups, one per compute unit
    a.lut_sat = pl->t.actSat;
    const size_t lds = r2c_wide_lds_bytes(g.nct, do_tanh, a.lut_sat);
    const int grid = (int)std::min<int64_t>(a.planes, (int64_t)pl->num_cu);
    hipError_t e = timed(kname, s, [&] {
      return launch_r2c_wide(a, g.nct, grid, lds, s);
    });
    if (e == hipSuccess) done = true;
    else if (e != hipErrorNotSupported) return hip_fail(e, kname);
  }
  if (!done || sigma) FNO_HIP(timed(kname, s, [&] { return launch_r2c(g.elem, g.nct, a, r2c_lds_bytes(g.elem, g.Kbp, g.R_f), s); }));
  if (g.nd == 3) {
    AxisArgs x{};
    x.in = inter;
    x.out = spec;
    x.er = pl->t.eFr;
    x.ei = pl->t.eFi;
    x.outer = g.B * C;
    x.Lin = g.N1;
    x.Lout = g.K1;
    x.inner = g.Ka * g.Kb;
    x.Linp = g.Linp_f;
    x.Lout16 = g.Lout16_f;
    x.scale = scale_mode == 0 ? (float)(1.0 / g.N1) : (float)(1.0 / std::sqrt((double)g.N1));
    FNO_HIP(timed("axis_fwd", s, [&] { return launch_axis(g.elem, x, axis_lds_bytes(g.elem, g.Linp_f), s); }));
  }
  return FNO_OK;
}

// Inverse: spectrum [B][C][K...] -> planes, out = scale * sum Re(Z e^{+i theta}).
fno_status run_c2r(const Plan* pl, const void* spec, void* out, void* inter, int64_t C,
                   float scale, const void* x_epi, hipStream_t s,
                   const double* bounds = nullptr) {
  const Geo& g = pl->g;
  const void* src = spec;
  if (g.nd == 3 && g.B * C > 65535) return FNO_ERR_UNSUPPORTED;
  if (g.nd == 3) {
    AxisArgs x{};
    x.in = spec;
    x.out = inter;
    x.er = pl->t.eIr;
    x.ei = pl->t.eIi;
    x.outer = g.B * C;
    x.Lin = g.K1;
    x.Lout = g.N1;
    x.inner = g.Ka * g.Kb;
    x.Linp = g.Linp_i;
    x.Lout16 = g.Lout16_i;
    x.scale = 1.0f;
    FNO_HIP(timed("axis_inv", s, [&] { return launch_axis(g.elem, x, axis_lds_bytes(g.elem, g.Linp_i), s); }));
    src = inter;
  }
  C2RArgs a{};
  a.zeros = pl->t.zeros;
  a.in = src;
  a.out = out;
  a.x = x_epi;
  a.cI = pl->t.cI;
  a.sI = pl->t.sI;
  a.twI = pl->t.twI;
  a.planes = g.B * C * (g.nd == 3 ? g.N1 : 1);
  a.Na = g.Na;
  a.Nb = g.Nb;
  a.Ka = g.Ka;
  a.Kb = g.Kb;
  a.Kbp = g.Kbp;
  a.Kap = g.Kap;
  a.Nap = g.Nap_i;
  a.R = g.R_i;
  a.scale = scale;
  a.epilogue = x_epi != nullptr;
  a.act = g.act;
  a.clip = g.clip;
  a.vec = (g.Nb % 8) == 0;
  if (a.planes > 0x7fffffff) return FNO_ERR_UNSUPPORTED;
  a.twIc = pl->t.twIc;
  a.cIc = pl->t.cIc;
  a.sIc = pl->t.sIc;
  a.lut = pl->t.lutGrad;
  const char* kname = !x_epi              ? "c2r_plane"
                      : g.act == ACT_TANH ? "c2r_plane_tanh_grad"
                      : g.act == ACT_CLIP ? "c2r_plane_clip_grad"
                                          : "c2r_plane_sigma_grad";
  if (x_epi && g.act == ACT_SIGMA) {
    // per-plane bounds, no table: the table-free kernel only
    if (!bounds) return FNO_ERR_INTERNAL;
    a.bounds = bounds;
    a.bgroup = g.nd == 3 ? g.N1 : 1;
    FNO_HIP(timed(kname, s, [&] { return launch_c2r(g.elem, g.nct, a, c2r_lds_bytes(g.elem, g.Kbp, g.Kap, g.R_i), s); }));
    return FNO_OK;
  }
  if (g.elem == ELEM_F16 && g.Nb % 16 == 0 && g.Kb % 4 == 0 && g.Nb <= 256 && g.Na <= 128) {
    const int ng = g.Nb64 / 64, ntb = g.Kbp / 16, nkz = g.Kap / 32;
    const size_t lds = c2r_chain_lds_bytes(ng, ntb, g.Kap, g.Na, x_epi != nullptr);
    const int64_t waves = (int64_t)kChainWaves;
    const int grid = (int)std::min<int64_t>((a.planes + waves - 1) / waves, (int64_t)2 * pl->num_cu);
    const size_t lut = x_epi ? 65536 : 0;  // static LDS of the kernel
    if (lds + lut <= 160 * 1024 && grid > 0 && c2r_chain_has(ng, ntb, nkz)) {
      hipError_t e = timed(kname, s, [&] { return launch_c2r_chain(a, ng, ntb, nkz, grid, lds, s); });
      if (e == hipSuccess) return FNO_OK;
      if (e != hipErrorNotSupported) return hip_fail(e, kname);
    }
  }
  if (g.elem == ELEM_F16 && a.vec && g.Kb % 4 == 0 && g.Nb <= 256 && g.Na <= 128 && g.nct <= 8 &&
      g.Kap <= 128) {
    const int nbt = (g.Nb + 63) / 64;
    const int nw = g.Na <= 64 ? 4 : 8;
    const int nkz = g.Kap / 32;
    const size_t lds = c2r_fast_lds_bytes(g.nct, nw, nbt, nkz);
    const int grid = (int)std::min<int64_t>(a.planes, (int64_t)2 * pl->num_cu);
    if (lds <= 80 * 1024) {
      hipError_t e = timed(kname, s, [&] {
        return launch_c2r_fast(a, g.nct, nw, nbt, nkz, grid, lds, s);
      });
      if (e == hipSuccess) return FNO_OK;
      if (e != hipErrorNotSupported) return hip_fail(e, kname);
    }
  }
  if (g.w2) {
    // large planes, one radix-2 stage per axis
    C2RArgs b = a;
    b.cI = pl->t.cI2;
    b.sI = pl->t.sI2;
    b.twI = pl->t.twI2;
    b.Kap = g.w2_kah;
    b.lut_sat = pl->t.gradSat;
    const size_t lds = c2r_wide2_lds_bytes(g.w2_nctc, g.w2_kah / 32, x_epi != nullptr, b.lut_sat);
    const int grid = (int)std::min<int64_t>(a.planes, (int64_t)pl->num_cu);
    hipError_t e = timed(kname, s, [&] { return launch_c2r_wide2(b, g.w2_nctc, grid, lds, s); });
    if (e == hipSuccess) return FNO_OK;
    if (e != hipErrorNotSupported) return hip_fail(e, kname);
  }
  if (g.elem == ELEM_F16 && g.Nb % 128 == 0 && g.Na % 256 == 0 &&
      (g.nct == 4 || g.nct == 8) && g.Kap <= 128 && g.Na * (int64_t)g.Nb * 2 < ((int64_t)1 << 30)) {
    // large planes: persistent eight-wave work-groups, one per compute unit
    a.lut_sat = pl->t.gradSat;
    const size_t lds = c2r_wide_lds_bytes(g.nct, g.Kap, x_epi != nullptr, a.lut_sat);
    const int grid = (int)std::min<int64_t>(a.planes, (int64_t)pl->num_cu);
    hipError_t e = timed(kname, s, [&] { return launch_c2r_wide(a, g.nct, grid, lds, s); });
    if (e == hipSuccess) return FNO_OK;
    if (e != hipErrorNotSupported) return hip_fail(e, kname);
  }
  FNO_HIP(timed(kname, s, [&] { return launch_c2r(g.elem, g.nct, a, c2r_lds_bytes(g.elem, g.Kbp, g.Kap, g.R_i), s); }));
  return FNO_OK;
}

fno_status run_contract(const Plan* pl, const void* in, const void* w, void* out,
                        bool adjoint, hipStream_t s) {
  const Geo& g = pl->g;
  ContractArgs a{};
  a.zeros = pl->t.zeros;
  a.in = in;
  a.w = w;
  a.out = out;
  a.B = (int)g.B;
  a.Q = (int)(adjoint ? g.Cout : g.Cin);
  a.P = (int)(adjoint ? g.Cin : g.Cout);
  a.K = (int)g.K;
  a.wrows = (int)g.Cin;
  a.wcols = (int)g.Cout;
  a.adjoint = adjoint;
  a.Kb = g.Kb;
  a.Nb = g.Nb;
  a.scale = 1.0f;
  if (g.K > 0x7fffffff / 2) return FNO_ERR_UNSUPPORTED;
  const bool slab = g.elem == ELEM_F16 && g.K % 16 == 0 && contract_slab_supported(a);
  FNO_HIP(timed(adjoint ? "contract_adjoint" : "contract", s, [&] {
    return slab ? launch_contract_slab(a, s) : launch_contract(g.elem, a, s);
  }));
  return FNO_OK;
}

// One pairwise Tucker step.  Operands carry labels, element type, conj flag.
struct Opnd {
  const void* ptr;
  std::string lab;
  int elem;
  int conj;
};

fno_status run_pair(const Sizes& sz, const Opnd& A0, const Opnd& B0, const std::string& res,
                    void* out, int out_elem, float scale, int c_axis_char, int Nb,
                    hipStream_t s, void* part = nullptr) {
  // the larger operand goes first (the kernels share its loads across a
  // result index it does not carry); the product commutes
  const bool swap = label_size(B0.lab, sz) > label_size(A0.lab, sz);
  const Opnd& A = swap ? B0 : A0;
  const Opnd& Bo = swap ? A0 : B0;
  PairArgs a{};
  a.a = A.ptr;
  a.b = Bo.ptr;
  a.out = out;
  a.a_elem = A.elem;
  a.b_elem = Bo.elem;
  a.conj_a = A.conj;
  a.conj_b = Bo.conj;
  a.out_elem = out_elem;
  auto strides = [&](const std::string& lab) {
    std::map<char, int64_t> st;
    int64_t acc = 1;
    for (int i = (int)lab.size() - 1; i >= 0; --i) {
      st[lab[i]] = acc;
      acc *= sz.at(lab[i]);
    }
    return st;
  };
  auto sa = strides(A.lab), sb = strides(Bo.lab);
  if ((int)res.size() > PW_MAXIDX) return FNO_ERR_UNSUPPORTED;
  a.n_out = (int)res.size();
  a.out_size = 1;
  a.scale_c_axis = -1;
  for (int k = 0; k < a.n_out; ++k) {
    char c = res[k];
    a.out_ext[k] = sz.at(c);
    a.out_size *= a.out_ext[k];
    a.a_stride_out[k] = sa.count(c) ? sa[c] : 0;
    a.b_stride_out[k] = sb.count(c) ? sb[c] : 0;
    if (c == c_axis_char) a.scale_c_axis = k;
  }
  std::string red;
  for (char c : A.lab + Bo.lab)
    if (res.find(c) == std::string::npos && red.find(c) == std::string::npos) red += c;
  if ((int)red.size() > PW_MAXIDX) return FNO_ERR_UNSUPPORTED;
  a.n_red = (int)red.size();
  a.red_size = 1;
  for (int k = 0; k < a.n_red; ++k) {
    char c = red[k];
    a.red_ext[k] = sz.at(c);
    a.red_size *= a.red_ext[k];
    a.a_stride_red[k] = sa.count(c) ? sa[c] : 0;
    a.b_stride_red[k] = sb.count(c) ? sb[c] : 0;
  }
  a.scale = scale;
  a.Nb = Nb;
  a.part = part;
  a.part_cap = part ? kPairPartBytes : 0;
  FNO_HIP(timed("tucker_pair", s, [&] { return launch_pair(a, s); }));
  return FNO_OK;
}

// Evaluate a Tucker or CP path: operands [spec, core (CP: lambda), u_in,
// u_out, u_1..u_d].
// Which steps of a factorised path a call runs: all of them; only those
// whose operands all come from the weights (no spectrum), which then take no
// split-K partial sums so that they may run beside the other steps; or the
// others, the first of them that reads a weights-only result waiting for the
// event `ready` (recorded after the weights-only steps on their stream).
enum PathSteps { PATH_ALL = 0, PATH_WEIGHTS = 1, PATH_REST = 2 };

// Whether a path has a step of the weights alone (operand 0 is the spectrum).
bool path_has_weight_steps(const std::vector<PStep>& path, size_t nops) {
  std::vector<char> wonly(nops, 1);
  wonly[0] = 0;
  for (const PStep& ps : path) {
    const char both = wonly[ps.p] && wonly[ps.q];
    if (both) return true;
    std::vector<char> next;
    for (int k = 0; k < (int)wonly.size(); ++k)
      if (k != ps.p && k != ps.q) next.push_back(wonly[k]);
    next.push_back(both);
    wonly.swap(next);
  }
  return false;
}

fno_status run_tucker_path(const fno_conv_desc* d, const Plan* pl, bool adjoint,
                           const void* spec, const fno_weights* w, void* out_spec,
                           char* scratch, hipStream_t s, int which = PATH_ALL,
                           hipEvent_t ready = nullptr) {
  const Geo& g = pl->g;
  Sizes sz = weight_sizes(d);
  const std::vector<PStep>& path = adjoint ? pl->path_adj : pl->path_fwd;
  const std::vector<std::string>& labs = adjoint ? pl->labels_adj : pl->labels_fwd;
  std::vector<Opnd> ops;
  ops.push_back({spec, labs[0], g.elem, 0});
  const int cj = adjoint ? 1 : 0;
  ops.push_back({w->core, labs[1], g.elem, cj});
  ops.push_back({w->u_in, labs[2], g.elem, cj});
  ops.push_back({w->u_out, labs[3], g.elem, cj});
  for (int j = 0; j < d->ndim; ++j) ops.push_back({w->u_mode[j], labs[4 + j], g.elem, cj});
  // split-K partial sums first, then one buffer per intermediate (sized for
  // fp32 complex).  Intermediates take the storage type: fp32 in the fp32
  // mode, fp16 in the half-precision mode, where the whole contraction runs
  // in half precision as the paper's mixed-precision layer does (products
  // exact in fp32 accumulators, each intermediate rounded once to fp16).
  void* part = scratch;
  size_t off = kPairPartBytes;
  const char clast = kSpatial[d->ndim - 1];
  // per operand: derived from the weights alone; produced by a weights-only
  // step (on the other stream when which == PATH_REST)
  std::vector<char> wonly(ops.size(), 1), made(ops.size(), 0);
  wonly[0] = 0;
  bool waited = ready == nullptr || which != PATH_REST;
  struct Join {  // the wait is enqueued on every way out
    bool& done;
    hipEvent_t ev;
    hipStream_t st;
    ~Join() {
      if (!done) (void)hipStreamWaitEvent(st, ev, 0);
    }
  } join{waited, ready, s};
  for (size_t st = 0; st < path.size(); ++st) {
    const PStep& ps = path[st];
    const bool last = st + 1 == path.size();
    const char wstep = wonly[ps.p] && wonly[ps.q];
    const bool run = which == PATH_ALL || (which == PATH_WEIGHTS) == (wstep != 0);
    void* dst;
    int oelem;
    if (last) {
      dst = out_spec;
      oelem = g.elem;
    } else {
      dst = scratch + off;
      off += (size_t)round_up(label_size(ps.res, sz) * 8, 256);
      oelem = g.elem;
    }
    // Storage order of an intermediate: the path's index order with the
    // last spatial index moved innermost where present, so that rows of the
    // spectrum stay contiguous (an outer product with the last axis' factor
    // would otherwise put the rank index, a few elements wide, innermost and
    // scatter the next step's loads).  The path itself is unchanged.
    std::string store = ps.res;
    if (!last) {
      const size_t pos = store.find(clast);
      if (pos != std::string::npos && pos + 1 != store.size()) {
        store.erase(pos, 1);
        store += clast;
      }
    }
    if (run) {
      if (!waited && (made[ps.p] || made[ps.q])) {
        const hipError_t e = hipStreamWaitEvent(s, ready, 0);
        waited = true;
        if (e != hipSuccess) return hip_fail(e, "wait for the weights-only steps");
      }
      fno_status r = run_pair(sz, ops[ps.p], ops[ps.q], store, dst, oelem, 1.0f,
                              last ? clast : 0, g.Nb, s, which == PATH_WEIGHTS ? nullptr : part);
      if (r != FNO_OK) return r;
    }
    std::vector<Opnd> next;
    std::vector<char> nw, nm;
    for (int k = 0; k < (int)ops.size(); ++k)
      if (k != ps.p && k != ps.q) {
        next.push_back(ops[k]);
        nw.push_back(wonly[k]);
        nm.push_back(made[k]);
      }
    next.push_back({dst, store, oelem, 0});
    nw.push_back(wstep);
    nm.push_back(wstep);
    ops.swap(next);
    wonly.swap(nw);
    made.swap(nm);
  }
  return FNO_OK;
}

// Phases of the factorised weight gradients: the steps that read only the
// weights (partial products of the core and the mode factors), and the
// steps that read the spectra.  Every phase lays out the scratch the same
// way, so the two may run as separate calls in order.
constexpr int WG_WEIGHTS = 1, WG_SPECTRA = 2, WG_ALL = 3;

// Extra streams of the spectrum phase.  After P and Q the chains of R (the
// core and mode-factor gradients), Z1 (g_u_in) and Z2 (g_u_out) read
// nothing the others write; with two more streams given, the Z1 and Z2
// chains run on them beside the R chain (forked on event pq after P and Q,
// joined back by d1 and d2).  Each chain has split-K partial sums of its
// own at the start of the scratch.
struct WgradBranches {
  hipStream_t z1, z2;
  hipEvent_t pq, d1, d2;
};
constexpr int kWgradChains = 3;

// Runs the Z1 and Z2 chains of a weight gradient on the streams of `br`
// (after the work already on s), or on s itself when br is null; joins them
// back to s when it goes out of scope.
struct WgradFork {
  hipStream_t s, z1, z2;
  const WgradBranches* br = nullptr;
  WgradFork(hipStream_t s_) : s(s_), z1(s_), z2(s_) {}
  fno_status fork(const WgradBranches* b) {
    if (!b) return FNO_OK;
    hipError_t e = hipEventRecord(b->pq, s);
    if (e == hipSuccess) e = hipStreamWaitEvent(b->z1, b->pq, 0);
    if (e != hipSuccess) return hip_fail(e, "fork of the weight-gradient chains");
    br = b;
    z1 = b->z1;
    e = hipStreamWaitEvent(b->z2, b->pq, 0);
    if (e != hipSuccess) return hip_fail(e, "fork of the weight-gradient chains");
    z2 = b->z2;
    return FNO_OK;
  }
  ~WgradFork() {
    if (z1 != s && hipEventRecord(br->d1, z1) == hipSuccess) (void)hipStreamWaitEvent(s, br->d1, 0);
    if (z2 != s && hipEventRecord(br->d2, z2) == hipSuccess) (void)hipStreamWaitEvent(s, br->d2, 0);
  }
  // split-K partial sums of the chain a step runs in
  char* part(char* scratch, hipStream_t st) const {
    return scratch + (st == z1 && z1 != s ? 1 : st == z2 && z2 != s ? 2 : 0) * kPairPartBytes;
  }
};

// Fixed schedule of the Tucker weight gradient (chain rule through the
// multilinear map): P = conj(Xhat u_in), Q = sqrt(N) c G conj(u_out),
// R = sum_b P Q, S = core x u_1 .. x u_d; g_core = R x conj(u_j)...,
// g_u_j = R . conj(core x_{q != j} u_q), g_u_in = conj(Xhat) . (Q conj S),
// g_u_out = (sqrt(N) c G) . (P conj S).  The weights-only steps (C_j, S)
// come first, then P and Q, then the three chains.
fno_status run_tucker_wgrad(const fno_conv_desc* d, const Plan* pl, const void* xh,
                            const void* gh, const fno_weights* w, fno_weight_grads* gw,
                            char* scratch, hipStream_t s, size_t* scratch_used = nullptr,
                            int phases = WG_ALL, const WgradBranches* br = nullptr) {
  const bool dry = scratch_used != nullptr;
  int phase = WG_WEIGHTS;  // the phase of the steps that follow
  WgradFork fk(s);
  auto run_pair = [&](const Sizes& sz_, const Opnd& A, const Opnd& Bo, const std::string& res,
                      void* out, int out_elem, float scale, int c_axis_char, int Nb,
                      hipStream_t st) -> fno_status {
    if (dry || !(phases & phase)) return FNO_OK;
    return fno::run_pair(sz_, A, Bo, res, out, out_elem, scale, c_axis_char, Nb, st,
                         fk.part(scratch, st));
  };
  const Geo& g = pl->g;
  const int nd = d->ndim;
  Sizes sz = tucker_sizes(d);
  std::string sp, rk;
  for (int j = 0; j < nd; ++j) {
    sp += kSpatial[j];
    rk += kRank[j];
  }
  const char clast = kSpatial[nd - 1];
  const float sqN = (float)std::sqrt((double)g.N);
  size_t off = kWgradChains * kPairPartBytes;  // split-K partial sums at the start
  auto buf = [&](const std::string& lab) {
    void* p = scratch + off;
    off += (size_t)round_up(label_size(lab, sz) * 8, 256);
    return p;
  };
  auto F = [&](const void* p, const std::string& lab, int conj) {
    return Opnd{p, lab, ELEM_F32, conj};
  };
  auto Wt = [&](const void* p, const std::string& lab, int conj) {
    return Opnd{p, lab, g.elem, conj};
  };
  auto U = [&](int j, int conj) {
    return Wt(w->u_mode[j], std::string(1, kSpatial[j]) + kRank[j], conj);
  };
  fno_status r;
  // ---- weights only ----
  // per-axis partial cores C_j = core x_{q != j} u_q, labels (a,e, r_j, sp\j)
  std::vector<Opnd> cj(nd);
  for (int j = 0; j < nd; ++j) {
    Opnd cur = Wt(w->core, "ae" + rk, 0);
    std::string lab = "ae" + rk;
    for (int q = 0; q < nd; ++q) {
      if (q == j) continue;
      std::string nl;
      for (char c : lab) nl += (c == kRank[q]) ? kSpatial[q] : c;
      void* dst = buf(nl);
      if ((r = run_pair(sz, cur, U(q, 0), nl, dst, ELEM_F32, 1.0f, 0, g.Nb, s))) return r;
      cur = F(dst, nl, 0);
      lab = nl;
    }
    cj[j] = Opnd{cur.ptr, cur.lab, cur.elem, 1};  // conjugated where it is read
  }
  // S[a,e,sp] = core x all u_j
  const std::string lS = "ae" + sp;
  void* S;
  {
    Opnd cur = Wt(w->core, "ae" + rk, 0);
    std::string lab = "ae" + rk;
    for (int q = 0; q < nd; ++q) {
      std::string nl;
      for (char c : lab) nl += (c == kRank[q]) ? kSpatial[q] : c;
      void* dst = buf(nl);
      if ((r = run_pair(sz, cur, U(q, 0), nl, dst, ELEM_F32, 1.0f, 0, g.Nb, s))) return r;
      cur = F(dst, nl, 0);
      lab = nl;
    }
    S = const_cast<void*>(cur.ptr);
  }
  // ---- spectra ----
  phase = WG_SPECTRA;
  const std::string lP = "ba" + sp, lQ = "be" + sp, lR = "ae" + sp;
  void* P = buf(lP);
  void* Q = buf(lQ);
  void* Rb = buf(lR);
  void* Z1 = buf("ba" + sp);
  void* Z2 = buf("be" + sp);
  // P[b,a,sp] = sum_i conj(Xhat[b,i,sp]) conj(u_in[i,a])
  r = run_pair(sz, Wt(xh, "bi" + sp, 1), Wt(w->u_in, "ia", 1), lP, P, ELEM_F32, 1.0f, 0, g.Nb, s);
  if (r) return r;
  // Q[b,e,sp] = sqrt(N) c(t) sum_o G[b,o,sp] conj(u_out[o,e])
  r = run_pair(sz, Wt(gh, "bo" + sp, 0), Wt(w->u_out, "oe", 1), lQ, Q, ELEM_F32, sqN, clast,
               g.Nb, s);
  if (r) return r;
  // R, Z1 and Z2 (below) in one launch where the ranks allow it
  bool tri = false;
  if (!dry && (phases & WG_SPECTRA)) {
    TriArgs ta{};
    ta.P = P;
    ta.Q = Q;
    ta.S = S;
    ta.R = Rb;
    ta.Z1 = Z1;
    ta.Z2 = Z2;
    ta.B = (int)sz['b'];
    ta.A = (int)sz['a'];
    ta.E = (int)sz['e'];
    ta.T = label_size(sp, sz);
    ta.scale = sqN;
    ta.c_ext = (int)sz[clast];
    ta.Nb = g.Nb;
    const hipError_t e = timed("tucker_pair", s, [&] { return launch_tucker_tri(ta, s); });
    if (e == hipSuccess) tri = true;
    else if (e != hipErrorNotSupported) return hip_fail(e, "tucker_tri");
  }
  if (!dry && (phases & WG_SPECTRA) && (r = fk.fork(br))) return r;
  // Z1[b,a,sp] = sum_e Q[b,e,sp] conj(S[a,e,sp]);  g_u_in = sum conj(Xhat) Z1
  if (!tri && (r = run_pair(sz, F(Q, lQ, 0), F(S, lS, 1), "ba" + sp, Z1, ELEM_F32, 1.0f, 0, g.Nb,
                            fk.z1)))
    return r;
  r = run_pair(sz, Wt(xh, "bi" + sp, 1), F(Z1, "ba" + sp, 0), "ia", gw->u_in, ELEM_F32, 1.0f, 0,
               g.Nb, fk.z1);
  if (r) return r;
  // Z2[b,e,sp] = sqrt(N) c(t) sum_a P[b,a,sp] conj(S[a,e,sp]); g_u_out = sum G Z2
  if (!tri && (r = run_pair(sz, F(P, lP, 0), F(S, lS, 1), "be" + sp, Z2, ELEM_F32, sqN, clast,
                            g.Nb, fk.z2)))
    return r;
  r = run_pair(sz, Wt(gh, "bo" + sp, 0), F(Z2, "be" + sp, 0), "oe", gw->u_out, ELEM_F32, 1.0f,
               0, g.Nb, fk.z2);
  if (r) return r;
  // R[a,e,sp] = sum_b P Q
  if (!tri && (r = run_pair(sz, F(P, lP, 0), F(Q, lQ, 0), lR, Rb, ELEM_F32, 1.0f, 0, g.Nb, s)))
    return r;
  // g_core[a,e,rk] = R contracted with conj(u_j) along every spatial axis
  {
    Opnd cur = F(Rb, lR, 0);
    std::string lab = lR;
    for (int j = 0; j < nd; ++j) {
      std::string nl;
      for (char c : lab) nl += (c == kSpatial[j]) ? kRank[j] : c;
      const bool last = j == nd - 1;
      void* dst = last ? gw->core : buf(nl);
      // reorder the final result to (a, e, rk)
      std::string res = last ? ("ae" + rk) : nl;
      if ((r = run_pair(sz, cur, U(j, 1), res, dst, ELEM_F32, 1.0f, 0, g.Nb, s))) return r;
      cur = F(dst, res, 0);
      lab = res;
    }
  }
  // g_u_j[x_j, r_j] = sum R[a,e,sp] conj(C_j[a,e,.., r_j, ..])
  for (int j = 0; j < nd; ++j) {
    std::string res = std::string(1, kSpatial[j]) + kRank[j];
    if ((r = run_pair(sz, F(Rb, lR, 0), cj[j], res, gw->u_mode[j], ELEM_F32, 1.0f, 0, g.Nb, s)))
      return r;
  }
  if (dry) *scratch_used = off;
  return FNO_OK;
}

size_t tucker_wgrad_bytes(const fno_conv_desc* d, const Plan* pl) {
  fno_weights w{};
  fno_weight_grads gw{};
  size_t used = 0;
  char dummy = 0;
  (void)run_tucker_wgrad(d, pl, &dummy, &dummy, &w, &gw, &dummy, nullptr, &used);
  return used;
}

// Fixed schedule of the CP weight gradient (chain rule through
// W = sum_r lambda_r u_in(r) u_out(r) prod_j u_j(r)), with G' = sqrt(N) c G:
//   P[b,r,sp] = sum_i conj(Xhat) conj(u_in),  Q[b,r,sp] = sum_o G' conj(u_out),
//   R[r,sp] = sum_b P Q,  S[r,sp] = lambda prod_j u_j,
//   g_lambda = sum_sp R prod_j conj(u_j),
//   g_u_j = conj(lambda) sum_{sp except j} R prod_{q != j} conj(u_q),
//   g_u_in = sum_{b,sp} conj(Xhat) (Q conj(S)),  g_u_out = sum_{b,sp} G' (P conj(S)).
fno_status run_cp_wgrad(const fno_conv_desc* d, const Plan* pl, const void* xh, const void* gh,
                        const fno_weights* w, fno_weight_grads* gw, char* scratch,
                        hipStream_t s, size_t* scratch_used = nullptr, int phases = WG_ALL,
                        const WgradBranches* br = nullptr) {
  const bool dry = scratch_used != nullptr;
  int phase = WG_WEIGHTS;  // the phase of the steps that follow
  WgradFork fk(s);
  auto pair = [&](const Sizes& sz_, const Opnd& A, const Opnd& Bo, const std::string& res,
                  void* out, float scale, int c_axis_char, hipStream_t st) -> fno_status {
    if (dry || !(phases & phase)) return FNO_OK;
    return run_pair(sz_, A, Bo, res, out, ELEM_F32, scale, c_axis_char, pl->g.Nb, st,
                    fk.part(scratch, st));
  };
  const Geo& g = pl->g;
  const int nd = d->ndim;
  Sizes sz = cp_sizes(d);
  std::string sp;
  for (int j = 0; j < nd; ++j) sp += kSpatial[j];
  const char clast = kSpatial[nd - 1];
  const float sqN = (float)std::sqrt((double)g.N);
  size_t off = kWgradChains * kPairPartBytes;  // split-K partial sums at the start
  auto buf = [&](const std::string& lab) {
    void* p = scratch + off;
    off += (size_t)round_up(label_size(lab, sz) * 8, 256);
    return p;
  };
  auto F = [&](const void* p, const std::string& lab, int conj) {
    return Opnd{p, lab, ELEM_F32, conj};
  };
  auto Wt = [&](const void* p, const std::string& lab, int conj) {
    return Opnd{p, lab, g.elem, conj};
  };
  auto U = [&](int j, int conj) { return Wt(w->u_mode[j], std::string(1, kSpatial[j]) + "r", conj); };
  fno_status r;
  // ---- weights only: S[r, sp] = lambda[r] prod_j u_j[sp_j, r] ----
  Opnd S = Wt(w->core, "r", 0);
  {
    std::string lab = "r";
    for (int j = 0; j < nd; ++j) {
      const std::string nl = lab + kSpatial[j];
      void* dst = buf(nl);
      if ((r = pair(sz, S, U(j, 0), nl, dst, 1.0f, 0, s))) return r;
      S = F(dst, nl, 0);
      lab = nl;
    }
  }
  const Opnd Sc{S.ptr, S.lab, S.elem, 1};
  // ---- spectra ----
  phase = WG_SPECTRA;
  const std::string lP = "br" + sp, lR = "r" + sp;
  void* P = buf(lP);
  void* Q = buf(lP);
  void* Rb = buf(lR);
  void* Z1 = buf(lP);
  void* Z2 = buf(lP);
  if ((r = pair(sz, Wt(xh, "bi" + sp, 1), Wt(w->u_in, "ir", 1), lP, P, 1.0f, 0, s))) return r;
  if ((r = pair(sz, Wt(gh, "bo" + sp, 0), Wt(w->u_out, "or", 1), lP, Q, sqN, clast, s))) return r;
  if (!dry && (phases & WG_SPECTRA) && (r = fk.fork(br))) return r;
  if ((r = pair(sz, F(Q, lP, 0), Sc, lP, Z1, 1.0f, 0, fk.z1))) return r;
  if ((r = pair(sz, Wt(xh, "bi" + sp, 1), F(Z1, lP, 0), "ir", gw->u_in, 1.0f, 0, fk.z1))) return r;
  if ((r = pair(sz, F(P, lP, 0), Sc, lP, Z2, sqN, clast, fk.z2))) return r;
  if ((r = pair(sz, Wt(gh, "bo" + sp, 0), F(Z2, lP, 0), "or", gw->u_out, 1.0f, 0, fk.z2)))
    return r;
  if ((r = pair(sz, F(P, lP, 0), F(Q, lP, 0), lR, Rb, 1.0f, 0, s))) return r;
  // g_lambda: contract R with conj(u_j) along every spatial axis
  {
    Opnd cur = F(Rb, lR, 0);
    std::string lab = lR;
    for (int j = 0; j < nd; ++j) {
      std::string nl;
      for (char c : lab)
        if (c != kSpatial[j]) nl += c;
      const bool last = j == nd - 1;
      void* dst = last ? gw->core : buf(nl);
      if ((r = pair(sz, cur, U(j, 1), nl, dst, 1.0f, 0, s))) return r;
      cur = F(dst, nl, 0);
      lab = nl;
    }
  }
  // g_u_j: R contracted with conj(u_q) for q != j, then times conj(lambda)
  for (int j = 0; j < nd; ++j) {
    Opnd cur = F(Rb, lR, 0);
    std::string lab = lR;
    for (int q = 0; q < nd; ++q) {
      if (q == j) continue;
      std::string nl;
      for (char c : lab)
        if (c != kSpatial[q]) nl += c;
      void* dst = buf(nl);
      if ((r = pair(sz, cur, U(q, 1), nl, dst, 1.0f, 0, s))) return r;
      cur = F(dst, nl, 0);
      lab = nl;
    }
    if ((r = pair(sz, cur, Wt(w->core, "r", 1), std::string(1, kSpatial[j]) + "r",
                  gw->u_mode[j], 1.0f, 0, s)))
      return r;
  }
  if (dry) *scratch_used = off;
  return FNO_OK;
}

size_t cp_wgrad_bytes(const fno_conv_desc* d, const Plan* pl) {
  fno_weights w{};
  fno_weight_grads gw{};
  size_t used = 0;
  char dummy = 0;
  (void)run_cp_wgrad(d, pl, &dummy, &dummy, &w, &gw, &dummy, nullptr, &used);
  return used;
}

fno_status check_weights(const fno_conv_desc* d, const fno_weights* w) {
  if (!w) return FNO_ERR_INVALID_ARGUMENT;
  if (d->weight_kind == FNO_WEIGHT_DENSE) {
    if (!w->dense || !aligned16(w->dense)) return FNO_ERR_INVALID_ARGUMENT;
  } else {
    if (!w->core || !w->u_in || !w->u_out) return FNO_ERR_INVALID_ARGUMENT;
    if (!aligned16(w->core) || !aligned16(w->u_in) || !aligned16(w->u_out))
      return FNO_ERR_INVALID_ARGUMENT;
    for (int j = 0; j < d->ndim; ++j)
      if (!w->u_mode[j] || !aligned16(w->u_mode[j])) return FNO_ERR_INVALID_ARGUMENT;
  }
  return FNO_OK;
}

inline bool okptr(const void* p) { return p && aligned16(p); }

// Workspace check from the host-only plan: runs before any device call.
fno_status check_ws(const fno_conv_desc* d, fno_op op, bool caches, const void* ws,
                    size_t ws_len) {
  Plan hp;
  host_plan(d, &hp);
  if (ws_len < ws_bytes(d, &hp, op, caches)) return FNO_ERR_WORKSPACE_TOO_SMALL;
  if (!okptr(ws)) return FNO_ERR_INVALID_ARGUMENT;
  return FNO_OK;
}

}  // namespace
}  // namespace fno

using namespace fno;

namespace fno {
fno_status report_hip_error(hipError_t e, const char* what) { return hip_fail(e, what); }

hipError_t timed_launch(const char* name, hipStream_t s, hipError_t (*launch)(void*), void* ctx) {
  return timed(name, s, [&] { return launch(ctx); });
}

// A second stream per device for work of one call that needs none of the
// other part's results: the factorised weight gradient of the combined
// backward (a chain of small, latency-bound contractions) runs on it while
// the caller's stream carries the transforms and the adjoint path.  The
// forks and the join are event waits, so the call stays ordered on the
// caller's stream as a whole (and a stream capture records both branches);
// calls that enqueue forks on one device take turns under a mutex.  Created
// on first use outside a stream capture and kept until the process ends.
struct SideStream {
  hipStream_t s = nullptr;
  hipEvent_t fork = nullptr, fork2 = nullptr, join = nullptr, ready = nullptr;
  // the weight gradient's own two extra chains
  hipStream_t z1 = nullptr, z2 = nullptr;
  hipEvent_t pq = nullptr, d1 = nullptr, d2 = nullptr;
  WgradBranches branches() const { return WgradBranches{z1, z2, pq, d1, d2}; }
};
std::mutex g_side_mutex;
std::map<int, SideStream> g_side;

// Whether work enqueued on `s` is being recorded into a graph.
bool capturing(hipStream_t s) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  return hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone;
}

// The device's side stream, or null (the caller then runs both parts on its
// own stream): when it cannot be created, or must not be because `s` is
// being captured.  Call with g_side_mutex held.
SideStream* side_stream_locked(hipStream_t s) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return nullptr;
  auto it = g_side.find(dev);
  if (it != g_side.end()) return &it->second;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess || cs != hipStreamCaptureStatusNone) return nullptr;
  SideStream ss;
  hipStream_t* st[3] = {&ss.s, &ss.z1, &ss.z2};
  hipEvent_t* ev[7] = {&ss.fork, &ss.fork2, &ss.join, &ss.ready, &ss.pq, &ss.d1, &ss.d2};
  bool ok = true;
  for (hipStream_t* p : st) ok = ok && hipStreamCreateWithFlags(p, hipStreamNonBlocking) == hipSuccess;
  for (hipEvent_t* e : ev) ok = ok && hipEventCreateWithFlags(e, hipEventDisableTiming) == hipSuccess;
  if (!ok) {
    for (hipEvent_t* e : ev)
      if (*e) (void)hipEventDestroy(*e);
    for (hipStream_t* p : st)
      if (*p) (void)hipStreamDestroy(*p);
    return nullptr;
  }
  return &(g_side[dev] = ss);
}

// Two branches after the work already on `s`: on the caller's stream
// first() then second(side); on the side stream side_a(side, stream), which
// reads nothing first() writes, and then side_b(stream), which reads
// first()'s results and nothing second() writes (second may wait for an
// event side_a records on the side stream; side is null when everything
// runs on `s`).  Everything enqueued on `s` afterwards follows both
// branches; the join is enqueued whatever the branches return.  Each part
// of the caller's work is enqueued before the side's, so that, launched
// from the host one by one, its few large kernels start while the side's
// many small ones are still being enqueued.
template <typename FA, typename F1, typename FB, typename F2>
fno_status run_forked(hipStream_t s, FA side_a, F1 first, FB side_b, F2 second) {
  std::unique_lock<std::mutex> lk(g_side_mutex);
  SideStream* ss = side_stream_locked(s);
  fno_status st;
  if (!ss) {
    lk.unlock();
    if ((st = first()) != FNO_OK || (st = second(nullptr)) != FNO_OK ||
        (st = side_a(nullptr, s)) != FNO_OK)
      return st;
    return side_b(s);
  }
  hipError_t e = hipEventRecord(ss->fork, s);
  if (e != hipSuccess) return hip_fail(e, "fork to the side stream");
  if ((st = first()) != FNO_OK) return st;  // nothing waits on the fork yet
  e = hipEventRecord(ss->fork2, s);
  if (e != hipSuccess) return hip_fail(e, "fork to the side stream");
  // side_a before second(): second() may wait on an event side_a records
  hipError_t ef = hipStreamWaitEvent(ss->s, ss->fork, 0);
  fno_status st_side = ef == hipSuccess ? side_a(ss, ss->s) : FNO_OK;
  const fno_status st_main = second(ef == hipSuccess ? ss : nullptr);
  if (ef == hipSuccess && st_side == FNO_OK) {
    ef = hipStreamWaitEvent(ss->s, ss->fork2, 0);
    if (ef == hipSuccess) st_side = side_b(ss->s);
  }
  const hipError_t ej = ef == hipSuccess ? hipEventRecord(ss->join, ss->s) : ef;
  const hipError_t ew = ej == hipSuccess ? hipStreamWaitEvent(s, ss->join, 0) : ej;
  if (st_side != FNO_OK) return st_side;
  if (st_main != FNO_OK) return st_main;
  return ew == hipSuccess ? FNO_OK : hip_fail(ew, "side stream");
}

// The weights-only steps of a factorised path on the side stream (recording
// ss->ready after them) when there are any; returns the event the rest of
// the path waits for, or null (then the caller's stream runs every step).
hipEvent_t path_weights_on_side(const fno_conv_desc* d, const Plan* pl, bool adjoint,
                                const fno_weights* w, char* scratch, SideStream* ss,
                                fno_status* st) {
  *st = FNO_OK;
  const std::vector<PStep>& path = adjoint ? pl->path_adj : pl->path_fwd;
  if (!ss || !path_has_weight_steps(path, 4 + (size_t)d->ndim)) return nullptr;
  *st = run_tucker_path(d, pl, adjoint, nullptr, w, nullptr, scratch, ss->s, PATH_WEIGHTS);
  const hipError_t e = hipEventRecord(ss->ready, ss->s);
  if (*st == FNO_OK && e != hipSuccess) *st = hip_fail(e, "side stream event");
  return *st == FNO_OK ? ss->ready : nullptr;
}

// A factorised path after its input transform(s): first() (the transforms)
// on the caller's stream, the path's weights-only steps on the side stream
// beside them, then the other steps on the caller's stream, waiting for the
// side before the first step that reads its results.  Everything on one
// stream when `allow_side` is false or the path has no weights-only step.
template <typename F1>
fno_status run_path_forked(const fno_conv_desc* d, const Plan* pl, bool adjoint,
                           const void* spec, const fno_weights* w, void* out, char* tsc,
                           hipStream_t s, bool allow_side, F1 first) {
  const std::vector<PStep>& path = adjoint ? pl->path_adj : pl->path_fwd;
  std::unique_lock<std::mutex> lk(g_side_mutex, std::defer_lock);
  SideStream* ss = nullptr;
  if (allow_side && path_has_weight_steps(path, 4 + (size_t)d->ndim)) {
    lk.lock();
    ss = side_stream_locked(s);
    if (!ss) lk.unlock();
  }
  hipError_t e = ss ? hipEventRecord(ss->fork, s) : hipSuccess;
  if (e != hipSuccess) return hip_fail(e, "fork to the side stream");
  fno_status st = first();
  if (st != FNO_OK) return st;  // nothing waits on the fork yet
  hipEvent_t ready = nullptr;
  if (ss) {
    e = hipStreamWaitEvent(ss->s, ss->fork, 0);
    if (e != hipSuccess) return hip_fail(e, "fork to the side stream");
    ready = path_weights_on_side(d, pl, adjoint, w, tsc, ss, &st);
    if (st != FNO_OK) {  // the side joins the caller's stream all the same
      if (hipEventRecord(ss->join, ss->s) == hipSuccess)
        (void)hipStreamWaitEvent(s, ss->join, 0);
      return st;
    }
  }
  return run_tucker_path(d, pl, adjoint, spec, w, out, tsc, s, ready ? PATH_REST : PATH_ALL,
                         ready);
}

// The forward call.  build_plan = false: the plan must already exist (no
// device allocation, no blocking upload; the allocation-free entry point).
fno_status fwd_impl(const fno_conv_desc* d, const void* x, const fno_weights* w, void* y,
                    void* x_hat_out, void* ws, size_t ws_len, hipStream_t s, bool build_plan) {
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  if (!okptr(x) || !okptr(y)) return FNO_ERR_INVALID_ARGUMENT;
  if (x_hat_out && !aligned16(x_hat_out)) return FNO_ERR_INVALID_ARGUMENT;
  if ((st = check_weights(d, w)) != FNO_OK) return st;
  if (build_plan && (st = check_ws(d, FNO_OP_FWD, true, ws, ws_len)) != FNO_OK) return st;
  std::shared_ptr<Plan> plan_ref;
  if ((st = get_plan(d, &plan_ref, build_plan)) != FNO_OK) return st;
  Plan* pl = plan_ref.get();
  if (!build_plan) {  // the cached plan gives the workspace size
    if (ws_len < ws_bytes(d, pl, FNO_OP_FWD, true)) return FNO_ERR_WORKSPACE_TOO_SMALL;
    if (!okptr(ws)) return FNO_ERR_INVALID_ARGUMENT;
  }
  const Geo& g = pl->g;
  WsLayout L;
  char* base = (char*)ws;
  char* xs = base + L.add(spec_bytes(g, g.Cin));
  char* ys = base + L.add(spec_bytes(g, g.Cout));
  char* inter = base + L.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
  char* tsc = base + L.total;
  double* bounds = (double*)(base + ws_core(d, pl, FNO_OP_FWD, true));
  void* xh = x_hat_out ? x_hat_out : (void*)xs;
  struct Flag {  // profiler events stay off for an allocation-free call
    bool prev;
    explicit Flag(bool on) : prev(g_no_alloc_call) { g_no_alloc_call = on; }
    ~Flag() { g_no_alloc_call = prev; }
  } flag(!build_plan);
  auto spectra = [&]() -> fno_status {
    fno_status r = run_sigma_stats(pl, x, bounds, s);
    return r != FNO_OK ? r : run_r2c(pl, x, xh, inter, g.Cin, 1, 0, s, bounds);
  };
  if (d->weight_kind == FNO_WEIGHT_DENSE) {
    if ((st = spectra()) != FNO_OK) return st;
    if ((st = run_contract(pl, xh, w->dense, ys, false, s)) != FNO_OK) return st;
  } else {
    // (the allocation-free call keeps to the caller's stream)
    st = run_path_forked(d, pl, false, xh, w, ys, tsc, s, build_plan, spectra);
    if (st != FNO_OK) return st;
  }
  return run_c2r(pl, ys, y, inter, g.Cout, 1.0f, nullptr, s);
}

}  // namespace fno

extern "C" {

const char* fno_last_error(void) { return g_last_error.c_str(); }

const char* fno_status_string(fno_status s) {
  switch (s) {
    case FNO_OK: return "FNO_OK";
    case FNO_ERR_INVALID_ARGUMENT: return "FNO_ERR_INVALID_ARGUMENT";
    case FNO_ERR_UNSUPPORTED: return "FNO_ERR_UNSUPPORTED";
    case FNO_ERR_WORKSPACE_TOO_SMALL: return "FNO_ERR_WORKSPACE_TOO_SMALL";
    case FNO_ERR_HIP: return "FNO_ERR_HIP";
    case FNO_ERR_INTERNAL: return "FNO_ERR_INTERNAL";
  }
  return "FNO_ERR_UNKNOWN";
}

fno_status fno_mode_frequency(const fno_conv_desc* d, int32_t axis, int64_t t, int64_t* k) {
  fno_status st = check_desc(d);
  if (st != FNO_OK && st != FNO_ERR_UNSUPPORTED) return st;
  if (!k || axis < 0 || axis >= d->ndim) return FNO_ERR_INVALID_ARGUMENT;
  const bool last = axis == d->ndim - 1;
  const int64_t ext = last ? d->modes[axis] : 2 * d->modes[axis];
  if (t < 0 || t >= ext) return FNO_ERR_INVALID_ARGUMENT;
  *k = mode_k(d->n[axis], d->modes[axis], last, t);
  return FNO_OK;
}

static fno_status path_for(const fno_conv_desc* d, fno_op op, std::vector<PStep>* path,
                           std::vector<std::string>* labs, std::string* out) {
  fno_status st = check_desc(d);
  if (st != FNO_OK && st != FNO_ERR_UNSUPPORTED) return st;
  if (!factorized(d)) return FNO_ERR_INVALID_ARGUMENT;
  if (op != FNO_OP_FWD && op != FNO_OP_BWD_DATA) return FNO_ERR_INVALID_ARGUMENT;
  weight_labels(d, op == FNO_OP_BWD_DATA, labs, out);
  *path = greedy_order(*labs, weight_sizes(d), *out, d->path_policy);
  return FNO_OK;
}

fno_status fno_contraction_path(const fno_conv_desc* d, fno_op op, int32_t* steps, int32_t cap,
                                int32_t* n_steps) {
  if (!n_steps) return FNO_ERR_INVALID_ARGUMENT;
  std::vector<PStep> path;
  std::vector<std::string> labs;
  std::string out;
  fno_status st = path_for(d, op, &path, &labs, &out);
  if (st != FNO_OK) return st;
  *n_steps = (int32_t)path.size();
  if (!steps || cap < (int32_t)path.size()) return FNO_ERR_INVALID_ARGUMENT;
  for (size_t i = 0; i < path.size(); ++i) {
    int32_t mask = 0;
    for (char c : path[i].res) mask |= 1 << label_bit(c);
    steps[3 * i] = path[i].p;
    steps[3 * i + 1] = path[i].q;
    steps[3 * i + 2] = mask;
  }
  return FNO_OK;
}

fno_status fno_contraction_path_cost(const fno_conv_desc* d, fno_op op, int64_t* macs,
                                     int64_t* peak) {
  if (!macs || !peak) return FNO_ERR_INVALID_ARGUMENT;
  std::vector<PStep> path;
  std::vector<std::string> labs;
  std::string out;
  fno_status st = path_for(d, op, &path, &labs, &out);
  if (st != FNO_OK) return st;
  Sizes sz = weight_sizes(d);
  int64_t total = 0, pk = 0;
  std::vector<std::string> ops = labs;
  for (const PStep& ps : path) {
    std::string both = ops[ps.p] + ops[ps.q];
    int64_t kred = 1;
    std::string seen;
    for (char c : both)
      if (ps.res.find(c) == std::string::npos && seen.find(c) == std::string::npos) {
        seen += c;
        kred *= sz.at(c);
      }
    const int64_t rs = label_size(ps.res, sz);
    total += rs * kred;
    pk = std::max(pk, rs);
    std::vector<std::string> next;
    for (int r = 0; r < (int)ops.size(); ++r)
      if (r != ps.p && r != ps.q) next.push_back(ops[r]);
    next.push_back(ps.res);
    ops.swap(next);
  }
  *macs = total;
  *peak = pk;
  return FNO_OK;
}

fno_status fno_spectrum_bytes(const fno_conv_desc* d, int which, size_t* bytes) {
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  if (!bytes || (which != 0 && which != 1)) return FNO_ERR_INVALID_ARGUMENT;
  const int64_t es = d->precision == FNO_PREC_FP16_TANH ? 2 : 4;
  const int64_t C = which == 0 ? d->c_in : d->c_out;
  *bytes = (size_t)(d->batch * C * kmodes(d) * 2 * es);
  return FNO_OK;
}

static fno_status ws_query(const fno_conv_desc* d, fno_op op, size_t* bytes, bool caches) {
  if (!bytes) return FNO_ERR_INVALID_ARGUMENT;
  if (op != FNO_OP_FWD && op != FNO_OP_BWD_DATA && op != FNO_OP_BWD_WEIGHT && op != FNO_OP_BWD)
    return FNO_ERR_INVALID_ARGUMENT;
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  Plan pl;
  host_plan(d, &pl);
  *bytes = ws_bytes(d, &pl, op, caches);
  return FNO_OK;
}

fno_status fno_spectral_conv_workspace_size(const fno_conv_desc* d, fno_op op, size_t* bytes) {
  return ws_query(d, op, bytes, true);
}

fno_status fno_spectral_conv_workspace_size_nocache(const fno_conv_desc* d, fno_op op,
                                                    size_t* bytes) {
  return ws_query(d, op, bytes, false);
}

fno_status fno_spectral_conv_fwd(const fno_conv_desc* d, const void* x, const fno_weights* w,
                                 void* y, void* x_hat_out, void* ws, size_t ws_len,
                                 hipStream_t s) {
  return fno::fwd_impl(d, x, w, y, x_hat_out, ws, ws_len, s, true);
}

fno_status fno_spectral_conv_bwd_data(const fno_conv_desc* d, const void* x,
                                      const fno_weights* w, const void* gy, void* gx,
                                      void* gy_hat_out, void* ws, size_t ws_len,
                                      hipStream_t s) {
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  const int pre_on = act_of(d) != ACT_NONE;  // x is read for f'(x)
  if (!okptr(gy) || !okptr(gx)) return FNO_ERR_INVALID_ARGUMENT;
  if (pre_on && !okptr(x)) return FNO_ERR_INVALID_ARGUMENT;
  if (gy_hat_out && !aligned16(gy_hat_out)) return FNO_ERR_INVALID_ARGUMENT;
  if ((st = check_weights(d, w)) != FNO_OK) return st;
  if ((st = check_ws(d, FNO_OP_BWD_DATA, true, ws, ws_len)) != FNO_OK) return st;
  std::shared_ptr<Plan> plan_ref;
  if ((st = get_plan(d, &plan_ref)) != FNO_OK) return st;
  Plan* pl = plan_ref.get();
  const Geo& g = pl->g;
  WsLayout L;
  char* base = (char*)ws;
  char* gs = base + L.add(spec_bytes(g, g.Cout));
  char* gxs = base + L.add(spec_bytes(g, g.Cin));
  char* inter = base + L.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
  char* tsc = base + L.total;
  double* bounds = (double*)(base + ws_core(d, pl, FNO_OP_BWD_DATA, true));
  void* gh = gy_hat_out ? gy_hat_out : (void*)gs;
  auto spectra = [&]() -> fno_status {
    fno_status r = run_sigma_stats(pl, x, bounds, s);
    return r != FNO_OK ? r : run_r2c(pl, gy, gh, inter, g.Cout, 0, 1, s);
  };
  if (d->weight_kind == FNO_WEIGHT_DENSE) {
    if ((st = spectra()) != FNO_OK) return st;
    if ((st = run_contract(pl, gh, w->dense, gxs, true, s)) != FNO_OK) return st;
  } else {
    if ((st = run_path_forked(d, pl, true, gh, w, gxs, tsc, s, true, spectra)) != FNO_OK)
      return st;
  }
  const float sc = (float)(1.0 / std::sqrt((double)g.N));
  return run_c2r(pl, gxs, gx, inter, g.Cin, sc, pre_on ? x : nullptr, s, bounds);
}

fno_status fno_spectral_conv_bwd_weight(const fno_conv_desc* d, const void* x, const void* gy,
                                        const fno_weights* w, const void* x_hat,
                                        const void* gy_hat, fno_weight_grads* gw, void* ws,
                                        size_t ws_len, hipStream_t s) {
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  if (!gw) return FNO_ERR_INVALID_ARGUMENT;
  if (x_hat ? !aligned16(x_hat) : !okptr(x)) return FNO_ERR_INVALID_ARGUMENT;
  if (gy_hat ? !aligned16(gy_hat) : !okptr(gy)) return FNO_ERR_INVALID_ARGUMENT;
  const bool tucker = factorized(d);
  if (tucker) {
    if ((st = check_weights(d, w)) != FNO_OK) return st;
    if (!okptr(gw->core) || !okptr(gw->u_in) || !okptr(gw->u_out))
      return FNO_ERR_INVALID_ARGUMENT;
    for (int j = 0; j < d->ndim; ++j)
      if (!okptr(gw->u_mode[j])) return FNO_ERR_INVALID_ARGUMENT;
  } else if (!okptr(gw->dense)) {
    return FNO_ERR_INVALID_ARGUMENT;
  }
  const bool caches = x_hat && gy_hat;
  if ((st = check_ws(d, FNO_OP_BWD_WEIGHT, caches, ws, ws_len)) != FNO_OK) return st;
  std::shared_ptr<Plan> plan_ref;
  if ((st = get_plan(d, &plan_ref)) != FNO_OK) return st;
  Plan* pl = plan_ref.get();
  const Geo& g = pl->g;
  WsLayout L;
  char* base = (char*)ws;
  const void* xh = x_hat;
  const void* gh = gy_hat;
  if (!caches) {
    char* xs = base + L.add(spec_bytes(g, g.Cin));
    char* gs = base + L.add(spec_bytes(g, g.Cout));
    char* inter = base + L.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
    if (!xh) {
      double* bounds = (double*)(base + ws_core(d, pl, FNO_OP_BWD_WEIGHT, false));
      if ((st = run_sigma_stats(pl, x, bounds, s)) != FNO_OK) return st;
      if ((st = run_r2c(pl, x, xs, inter, g.Cin, 1, 0, s, bounds)) != FNO_OK) return st;
      xh = xs;
    }
    if (!gh) {
      if ((st = run_r2c(pl, gy, gs, inter, g.Cout, 0, 1, s)) != FNO_OK) return st;
      gh = gs;
    }
  }
  char* tsc = base + L.total;
  if (!tucker) {
    WgradArgs a{};
    a.zeros = pl->t.zeros;
    a.xh = xh;
    a.gh = gh;
    a.gw = (float*)gw->dense;
    a.B = (int)g.B;
    a.Cin = (int)g.Cin;
    a.Cout = (int)g.Cout;
    a.K = (int)g.K;
    a.Kb = g.Kb;
    a.Nb = g.Nb;
    a.scale = (float)std::sqrt((double)g.N);
    const bool slab = g.elem == ELEM_F16 && g.K % 16 == 0 && wgrad_slab_supported(a);
    FNO_HIP(timed("wgrad", s, [&] {
      return slab ? launch_wgrad_slab(a, s) : launch_wgrad(g.elem, a, s);
    }));
    return FNO_OK;
  }
  // the chains after P and Q on the side streams when they exist
  std::unique_lock<std::mutex> lk(g_side_mutex);
  SideStream* ss = capturing(s) ? nullptr : side_stream_locked(s);
  WgradBranches wb{};
  if (ss) wb = ss->branches();
  const WgradBranches* b = ss ? &wb : nullptr;
  if (d->weight_kind == FNO_WEIGHT_CP)
    return run_cp_wgrad(d, pl, xh, gh, w, gw, tsc, s, nullptr, WG_ALL, b);
  return run_tucker_wgrad(d, pl, xh, gh, w, gw, tsc, s, nullptr, WG_ALL, b);
}

fno_status fno_spectral_conv_bwd(const fno_conv_desc* d, const void* x, const fno_weights* w,
                                 const void* gy, const void* x_hat, void* gx,
                                 fno_weight_grads* gw, void* gy_hat_out, void* ws,
                                 size_t ws_len, hipStream_t s) {
  fno_status st = check_desc(d);
  if (st != FNO_OK) return st;
  const int pre_on = act_of(d) != ACT_NONE;  // x is read for f'(x)
  const bool tucker = factorized(d);
  if (!okptr(gy) || !okptr(gx) || !gw) return FNO_ERR_INVALID_ARGUMENT;
  if ((pre_on || !x_hat) && !okptr(x)) return FNO_ERR_INVALID_ARGUMENT;
  if (x_hat && !aligned16(x_hat)) return FNO_ERR_INVALID_ARGUMENT;
  if (gy_hat_out && !aligned16(gy_hat_out)) return FNO_ERR_INVALID_ARGUMENT;
  if ((st = check_weights(d, w)) != FNO_OK) return st;
  if (tucker) {
    if (!okptr(gw->core) || !okptr(gw->u_in) || !okptr(gw->u_out))
      return FNO_ERR_INVALID_ARGUMENT;
    for (int j = 0; j < d->ndim; ++j)
      if (!okptr(gw->u_mode[j])) return FNO_ERR_INVALID_ARGUMENT;
  } else if (!okptr(gw->dense)) {
    return FNO_ERR_INVALID_ARGUMENT;
  }
  const bool cache = x_hat != nullptr;
  if ((st = check_ws(d, FNO_OP_BWD, cache, ws, ws_len)) != FNO_OK) return st;
  std::shared_ptr<Plan> plan_ref;
  if ((st = get_plan(d, &plan_ref)) != FNO_OK) return st;
  Plan* pl = plan_ref.get();
  const Geo& g = pl->g;
  WsLayout L;
  char* base = (char*)ws;
  char* gs = base + L.add(spec_bytes(g, g.Cout));
  char* xs = cache ? nullptr : base + L.add(spec_bytes(g, g.Cin));
  char* wsd = base + L.add(ws_bytes(d, pl, FNO_OP_BWD_DATA, true));
  void* gh = gy_hat_out ? gy_hat_out : (void*)gs;
  if (tucker) {
    // the data part's regions inside wsd, laid out as in bwd_data (its first
    // region, the gradient spectrum, is unused: gh holds it), then the
    // weight part's scratch
    char* wsw = base + L.add(ws_bytes(d, pl, FNO_OP_BWD_WEIGHT, true));
    WsLayout Ld;
    (void)Ld.add(spec_bytes(g, g.Cout));
    char* gxs = wsd + Ld.add(spec_bytes(g, g.Cin));
    char* inter = wsd + Ld.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
    char* tsc = wsd + Ld.total;
    double* bounds = (double*)(wsd + ws_core(d, pl, FNO_OP_BWD_DATA, true));
    const void* xh = x_hat ? x_hat : (const void*)xs;
    // The weight gradient writes only its own scratch and gw; its steps
    // that read only the weights run beside the transforms of gy (and x),
    // the rest beside the adjoint path and the inverse transform.
    WgradBranches wb{};
    auto wgrad = [&](int phases, hipStream_t st_, const WgradBranches* b) {
      return d->weight_kind == FNO_WEIGHT_CP
                 ? run_cp_wgrad(d, pl, xh, gh, w, gw, wsw, st_, nullptr, phases, b)
                 : run_tucker_wgrad(d, pl, xh, gh, w, gw, wsw, st_, nullptr, phases, b);
    };
    // the side first takes the adjoint path's weights-only steps, which the
    // caller's stream waits for before the first step that reads them
    hipEvent_t ready = nullptr;
    const WgradBranches* pwb = nullptr;
    auto side_a = [&](SideStream* ss, hipStream_t st_) {
      fno_status r;
      ready = path_weights_on_side(d, pl, true, w, tsc, ss, &r);
      // The weight gradient's Z1 and Z2 chains run on the caller's stream
      // after its inverse transform (which it enqueues first), beside the
      // side stream's R chain: the caller's stream waits for P, Q and the
      // fused products on the side stream, and the side stream for the
      // chains.  (Forking the chains off the side stream onto two more
      // streams instead ended the process inside the runtime's
      // end-of-capture call under a stream capture, cause not found, and
      // was no faster when launched from the host.)
      if (ss) {
        wb = ss->branches();
        wb.z1 = wb.z2 = s;
        pwb = &wb;
      }
      return r != FNO_OK ? r : wgrad(WG_WEIGHTS, st_, nullptr);
    };
    auto side_b = [&](hipStream_t st_) { return wgrad(WG_SPECTRA, st_, pwb); };
    auto spectra = [&]() -> fno_status {
      fno_status r = run_sigma_stats(pl, x, bounds, s);
      if (r == FNO_OK) r = run_r2c(pl, gy, gh, inter, g.Cout, 0, 1, s);
      if (r == FNO_OK && !cache) r = run_r2c(pl, x, xs, inter, g.Cin, 1, 0, s, bounds);
      return r;
    };
    auto data_part = [&](SideStream*) -> fno_status {
      fno_status r = run_tucker_path(d, pl, true, gh, w, gxs, tsc, s,
                                     ready ? PATH_REST : PATH_ALL, ready);
      if (r != FNO_OK) return r;
      const float sc = (float)(1.0 / std::sqrt((double)g.N));
      return run_c2r(pl, gxs, gx, inter, g.Cin, sc, pre_on ? x : nullptr, s, bounds);
    };
    return run_forked(s, side_a, spectra, side_b, data_part);
  }
  // dense: the data part's regions inside wsd, laid out as in bwd_data (its
  // first region, the gradient spectrum, is unused: gh holds it)
  WsLayout Ld;
  (void)Ld.add(spec_bytes(g, g.Cout));
  char* gxs = wsd + Ld.add(spec_bytes(g, g.Cin));
  char* inter = wsd + Ld.add(std::max(inter3d_bytes(g, g.Cin), inter3d_bytes(g, g.Cout)));
  double* bounds = (double*)(wsd + ws_core(d, pl, FNO_OP_BWD_DATA, true));
  if (pre_on && (st = run_sigma_stats(pl, x, bounds, s)) != FNO_OK) return st;
  const void* xh = x_hat;
  if (!cache) {
    if ((st = run_r2c(pl, x, xs, inter, g.Cin, 1, 0, s, bounds)) != FNO_OK) return st;
    xh = xs;
  }
  if ((st = run_r2c(pl, gy, gh, inter, g.Cout, 0, 1, s)) != FNO_OK) return st;
  ContractArgs a{};
  a.zeros = pl->t.zeros;
  a.in = gh;
  a.w = w->dense;
  a.out = gxs;
  a.B = (int)g.B;
  a.Q = (int)g.Cout;
  a.P = (int)g.Cin;
  a.K = (int)g.K;
  a.wrows = (int)g.Cin;
  a.wcols = (int)g.Cout;
  a.adjoint = 1;
  a.Kb = g.Kb;
  a.Nb = g.Nb;
  a.scale = 1.0f;
  WgradArgs wa{};
  wa.zeros = pl->t.zeros;
  wa.xh = xh;
  wa.gh = gh;
  wa.gw = (float*)gw->dense;
  wa.B = (int)g.B;
  wa.Cin = (int)g.Cin;
  wa.Cout = (int)g.Cout;
  wa.K = (int)g.K;
  wa.Kb = g.Kb;
  wa.Nb = g.Nb;
  wa.scale = (float)std::sqrt((double)g.N);
  if (g.elem == ELEM_F16 && g.K <= 0x7fffffff / 2 && adj_wgrad_slab_supported(a, wa)) {
    FNO_HIP(timed("contract_adjoint_wgrad", s, [&] { return launch_adj_wgrad_slab(a, wa, s); }));
  } else {
    if ((st = run_contract(pl, gh, w->dense, gxs, true, s)) != FNO_OK) return st;
    const bool slab = g.elem == ELEM_F16 && g.K % 16 == 0 && wgrad_slab_supported(wa);
    FNO_HIP(timed("wgrad", s, [&] {
      return slab ? launch_wgrad_slab(wa, s) : launch_wgrad(g.elem, wa, s);
    }));
  }
  const float sc = (float)(1.0 / std::sqrt((double)g.N));
  return run_c2r(pl, gxs, gx, inter, g.Cin, sc, pre_on ? x : nullptr, s, bounds);
}

fno_status fno_profile_enable(int32_t enable) {
  std::lock_guard<std::mutex> lk(g_prof_mutex);
  g_prof_on = enable != 0;
  return FNO_OK;
}

fno_status fno_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_prof_mutex);
  prof_drain();
  g_prof.clear();
  return FNO_OK;
}

fno_status fno_profile_read(int32_t index, char* name, int32_t name_cap, int64_t* launches,
                            double* total_ms) {
  std::lock_guard<std::mutex> lk(g_prof_mutex);
  prof_drain();
  if (index < 0 || index >= (int32_t)g_prof.size()) return FNO_ERR_INVALID_ARGUMENT;
  const ProfEntry& e = g_prof[index];
  if (name && name_cap > 0) {
    std::strncpy(name, e.name.c_str(), (size_t)name_cap - 1);
    name[name_cap - 1] = 0;
  }
  if (launches) *launches = e.launches;
  if (total_ms) *total_ms = e.total_ms;
  return FNO_OK;
}

fno_status fno_release_caches(void) {
  std::map<PlanKey, std::shared_ptr<Plan>> gone;
  {
    std::lock_guard<std::mutex> lock(g_mutex);
    gone.swap(g_plans);
  }
  // plans no call holds are destroyed here (their tables freed); a plan in
  // use by a call on another thread goes when that call returns
  gone.clear();
  return FNO_OK;
}

}  // extern "C"
