// Expert grouping and adapter consolidation: Sec. 3.3 (rank consolidation)
// with the appendices on the layer-wise similarity graph, Louvain grouping
// and group anchors.
//
// Host (E <= 256 nodes; microseconds, no device work):
//   similarity graph -- W_ij = max(0, sym(S)_ij - b) off the diagonal, b the
//                       median of the off-diagonal entries of sym(S) =
//                       (S + S^T) / 2; zero diagonal
//   Louvain          -- greedy local moves on the weighted modularity
//                       Q = (1/2m) sum_ij (W_ij - gamma k_i k_j / 2m)[z_i = z_j]:
//                       node i (index order) leaves its community and joins
//                       the candidate (a neighbour's community or its own)
//                       with the largest gain k_i,in(C) - gamma k_i tot(C)/2m,
//                       ties to the lowest community id, only if that gain
//                       beats staying; sweeps until none moves, then the
//                       communities become super-nodes; ends at a level with
//                       no move.  Degrees, 2m, k_i,in and coarse weights are
//                       summed in index order, so the partition is
//                       reproducible bit for bit.
//   anchors          -- the CKA centre of a group: the member with the largest
//                       summed similarity to the other members (ties to the
//                       lowest index)
// Device:
//   consolidate      -- group adapters from the expert adapters: rank rows
//                       0 .. r-1 of A_g = A_anchor, columns 0 .. r-1 of B_g =
//                       (r_g / r) B_anchor (the group adapter at alpha / r_g
//                       reproduces the anchor's update), the other rows of A_g
//                       from the caller's standard-init draw, the other
//                       columns of B_g zero.
#include <algorithm>
#include <numeric>
#include <vector>

#include "ace_device.hpp"
#include "ace_internal.hpp"

namespace ace {

namespace {

void degrees(const std::vector<double>& W, int n, std::vector<double>& k, double& two_m) {
  k.assign(n, 0.0);
  for (int i = 0; i < n; ++i) {
    double s = 0.0;
    for (int j = 0; j < n; ++j) s += W[(size_t)i * n + j];
    k[i] = s;
  }
  two_m = 0.0;
  for (int i = 0; i < n; ++i) two_m += k[i];
}

// One level of local moves from singletons; false when no node moved.
bool local_moves(const std::vector<double>& W, int n, double gamma, std::vector<int>& comm) {
  std::vector<double> k;
  double two_m;
  degrees(W, n, k, two_m);
  comm.resize(n);
  std::iota(comm.begin(), comm.end(), 0);
  if (!(two_m > 0.0)) return false;
  std::vector<double> tot(k), kin(n, 0.0);
  std::vector<char> seen(n, 0);
  std::vector<int> touched;
  touched.reserve(n);
  bool moved_any = false;
  for (;;) {
    bool moved = false;
    for (int i = 0; i < n; ++i) {
      const int ci = comm[i];
      tot[ci] -= k[i];
      touched.clear();
      for (int j = 0; j < n; ++j) {
        const double w = W[(size_t)i * n + j];
        if (j != i && w > 0.0) {
          const int c = comm[j];
          if (!seen[c]) {
            seen[c] = 1;
            kin[c] = 0.0;
            touched.push_back(c);
          }
          kin[c] += w;
        }
      }
      auto gain = [&](int c) {
        const double kc = seen[c] ? kin[c] : 0.0;
        return kc - gamma * k[i] * tot[c] / two_m;
      };
      int best = ci;
      double gbest = gain(ci);
      for (int c : touched) {
        const double gc = gain(c);
        if (gc > gbest || (gc == gbest && c < best)) {
          best = c;
          gbest = gc;
        }
      }
      if (best != ci && gbest > gain(ci)) {
        comm[i] = best;
        moved = true;
        moved_any = true;
      }
      tot[comm[i]] += k[i];
      for (int c : touched) seen[c] = 0;
    }
    if (!moved) break;
  }
  return moved_any;
}

// Relabels in order of first appearance; returns the number of labels.
int renumber(std::vector<int>& z) {
  std::vector<int> map(z.size(), -1);
  int next = 0;
  for (int& v : z) {
    if (map[v] < 0) map[v] = next++;
    v = map[v];
  }
  return next;
}

// ---------------------------------------------------------------- device

struct ConsolidateArgs {
  const void* A;        // [E*r][d_in]
  const void* B;        // expert e: [d_out][r] at d_out * r * e
  const void* A_init;   // [(E - G) * r][d_in]
  void* Ag;             // [R][d_in], group blocks in group order
  void* Bg;             // group g: [d_out][r_g] at d_out * roff_g
  int32_t d_in, d_out, r;
  KeyTable keys;        // group ranks r_g and offsets roff_g
  uint8_t anchor[kMaxKeys];
};

// Block b copies row b of A_g (16-byte pieces).
template <typename T>
__global__ __launch_bounds__(kThreads) void consolidate_a_kernel(ConsolidateArgs a) {
  using F = typename Tr<T>::frag;
  constexpr int PER = Tr<T>::PER;
  const int row = blockIdx.x;
  const int g = upper_index(a.keys.roff, a.keys.n_keys, row);
  const int rho = row - a.keys.roff[g];
  const T* src = rho < a.r
      ? static_cast<const T*>(a.A) + ((size_t)a.anchor[g] * a.r + rho) * a.d_in
      : static_cast<const T*>(a.A_init) + ((size_t)(a.keys.roff[g] - g * a.r) + rho - a.r) * a.d_in;
  T* dst = static_cast<T*>(a.Ag) + (size_t)row * a.d_in;
  for (int c = threadIdx.x * PER; c < a.d_in; c += kThreads * PER)
    Tr<T>::store(dst + c, Tr<T>::load(src + c));
}

// Element t of B_g (grid-stride over R * d_out elements).
template <typename T>
__global__ __launch_bounds__(kThreads) void consolidate_b_kernel(ConsolidateArgs a) {
  const long total = (long)a.keys.R * a.d_out;
  const T* B = static_cast<const T*>(a.B);
  T* Bg = static_cast<T*>(a.Bg);
  for (long t = (long)blockIdx.x * kThreads + threadIdx.x; t < total; t += (long)gridDim.x * kThreads) {
    const int g = upper_index(a.keys.roff, a.keys.n_keys, (int)(t / a.d_out));
    const long base = (long)a.d_out * a.keys.roff[g];
    const int rg = a.keys.rank[g];
    const long loc = t - base;
    const int o = (int)(loc / rg), rho = (int)(loc % rg);
    float v = 0.f;
    if (rho < a.r)
      v = (float)(rg / a.r) * (float)B[(size_t)a.d_out * a.r * a.anchor[g] + (size_t)o * a.r + rho];
    Bg[t] = (T)v;
  }
}

template <typename T>
hipError_t launch_consolidate_t(const ConsolidateArgs& a, hipStream_t stream) {
  if (a.keys.R > 0) consolidate_a_kernel<T><<<a.keys.R, kThreads, 0, stream>>>(a);
  const long total = (long)a.keys.R * a.d_out;
  const long blocks = std::min<long>((total + kThreads - 1) / kThreads, 8L * device_cu_count());
  if (blocks > 0) consolidate_b_kernel<T><<<(int)blocks, kThreads, 0, stream>>>(a);
  return hipGetLastError();
}

}  // namespace

void similarity_graph(const float* S, int E, double* W) {
  std::vector<double> sym((size_t)E * E, 0.0);
  std::vector<double> off;
  off.reserve((size_t)E * (E > 0 ? E - 1 : 0));
  for (int i = 0; i < E; ++i)
    for (int j = 0; j < E; ++j)
      if (i != j) {
        const double v = ((double)S[(size_t)i * E + j] + (double)S[(size_t)j * E + i]) / 2.0;
        sym[(size_t)i * E + j] = v;
        off.push_back(v);
      }
  double b = 0.0;
  if (!off.empty()) {
    std::sort(off.begin(), off.end());
    const size_t m = off.size();
    b = (m % 2) ? off[m / 2] : (off[m / 2 - 1] + off[m / 2]) / 2.0;
  }
  for (int i = 0; i < E; ++i)
    for (int j = 0; j < E; ++j)
      W[(size_t)i * E + j] = (i == j || E < 2) ? 0.0 : std::max(0.0, sym[(size_t)i * E + j] - b);
}

int louvain(const double* W, int E, double gamma, int32_t* groups) {
  std::vector<double> Wl(W, W + (size_t)E * E);
  int nl = E;
  std::vector<int> node_of(E);
  std::iota(node_of.begin(), node_of.end(), 0);
  for (;;) {
    std::vector<int> comm;
    if (!local_moves(Wl, nl, gamma, comm)) break;
    const int nc = renumber(comm);
    std::vector<double> Wc((size_t)nc * nc, 0.0);
    for (int i = 0; i < nl; ++i)
      for (int j = 0; j < nl; ++j) Wc[(size_t)comm[i] * nc + comm[j]] += Wl[(size_t)i * nl + j];
    Wl.swap(Wc);
    nl = nc;
    for (int& v : node_of) v = comm[v];
  }
  const int G = renumber(node_of);
  for (int e = 0; e < E; ++e) groups[e] = node_of[e];
  return G;
}

void group_anchors(const float* S, int E, const int32_t* e2g, int G, int32_t* anchors) {
  for (int g = 0; g < G; ++g) {
    int best = -1;
    double best_score = 0.0;
    for (int i = 0; i < E; ++i) {
      if (e2g[i] != g) continue;
      double score = 0.0;
      for (int j = 0; j < E; ++j)
        if (j != i && e2g[j] == g) score += (double)S[(size_t)i * E + j];
      if (best < 0 || score > best_score) {
        best = i;
        best_score = score;
      }
    }
    anchors[g] = best;
  }
}

hipError_t launch_consolidate(int dtype, const ConsolidateProblem& p, hipStream_t stream) {
  ConsolidateArgs a{};
  a.A = p.A;
  a.B = p.B;
  a.A_init = p.A_init;
  a.Ag = p.Ag;
  a.Bg = p.Bg;
  a.d_in = p.d_in;
  a.d_out = p.d_out;
  a.r = p.r;
  a.keys = p.keys;
  for (int g = 0; g < p.keys.n_keys; ++g) a.anchor[g] = (uint8_t)p.anchor[g];
  if (dtype == ACE_BF16) return launch_consolidate_t<__bf16>(a, stream);
  return launch_consolidate_t<float>(a, stream);
}

}  // namespace ace
