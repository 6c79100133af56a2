// Host construction of the library's dense +-1 Hadamard factors (orders 1, 28, 172).
//
// The online rotations R3/R4 of Sec. 3.1 are Hadamard matrices; for widths that are
// not powers of two the rotation is H_a (x) S_b with a small dense factor H_a.  The
// paper does not say which Hadamard matrix of order 28 or 172; any one is valid.
//   order 28 : Paley type II from the prime q = 13 (q = 1 mod 4):
//              H = C (x) [[1,1],[1,-1]] + I (x) [[1,-1],[-1,-1]],
//              C = [[0, 1^T], [1, Q]], Q[i][j] = chi(j - i), chi the quadratic character.
//   order 172: Williamson array [[A,B,C,D],[-B,A,-D,C],[-C,D,A,-B],[-D,-C,B,A]] from four
//              symmetric circulants of order 43 whose periodic autocorrelations sum to
//              zero off the origin.  First rows are constant on the cosets of the
//              order-6 subgroup of (Z/43)^* (it contains -1, so the circulants are
//              symmetric); candidate t has sign (-1)^bit0(t) at index 0 and
//              (-1)^bit(j+1)(t) on coset g^j G (g the least primitive root).  The
//              quadruple used is the first in lexicographic order of (tA,tB,tC,tD) with
//              tA <= tB <= tC <= tD.
#include <cstdint>
#include <map>
#include <vector>

#include "sq_internal.h"

namespace sq {
namespace {

bool is_prime(int q) {
  if (q < 2) return false;
  for (int d = 2; d * d <= q; ++d)
    if (q % d == 0) return false;
  return true;
}

int powmod(int b, int e, int m) {
  long long r = 1, x = b % m;
  while (e) {
    if (e & 1) r = r * x % m;
    x = x * x % m;
    e >>= 1;
  }
  return static_cast<int>(r);
}

std::vector<int8_t> paley2(int q) {
  std::vector<int> chi(q, -1);
  chi[0] = 0;
  for (int x = 1; x < q; ++x) chi[(x * x) % q] = 1;
  const int c = q + 1;
  std::vector<int> conf(c * c, 0);
  for (int j = 1; j < c; ++j) conf[j] = 1, conf[j * c] = 1;
  for (int i = 0; i < q; ++i)
    for (int j = 0; j < q; ++j) conf[(i + 1) * c + (j + 1)] = chi[((j - i) % q + q) % q];
  const int n = 2 * c;
  static const int P[2][2] = {{1, 1}, {1, -1}};
  static const int Q[2][2] = {{1, -1}, {-1, -1}};
  std::vector<int8_t> h(n * n);
  for (int i = 0; i < c; ++i)
    for (int j = 0; j < c; ++j)
      for (int s = 0; s < 2; ++s)
        for (int t = 0; t < 2; ++t)
          h[(2 * i + s) * n + (2 * j + t)] =
              static_cast<int8_t>(conf[i * c + j] * P[s][t] + (i == j ? Q[s][t] : 0));
  return h;
}

std::vector<int8_t> williamson(int m, int sub_order) {
  int g = 0;
  for (int cand = 2; cand < m && !g; ++cand) {
    bool prim = true;
    for (int p = 2; p < m; ++p)
      if ((m - 1) % p == 0 && is_prime(p) && powmod(cand, (m - 1) / p, m) == 1) prim = false;
    if (prim) g = cand;
  }
  const int ncos = (m - 1) / sub_order;
  const int hgen = powmod(g, ncos, m);
  std::vector<int> coset(m, -1);
  for (int j = 0; j < ncos; ++j)
    for (int k = 0; k < sub_order; ++k)
      coset[(static_cast<long long>(powmod(g, j, m)) * powmod(hgen, k, m)) % m] = j;
  const int ncand = 1 << (ncos + 1);
  std::vector<std::vector<int>> rows(ncand, std::vector<int>(m));
  for (int t = 0; t < ncand; ++t) {
    rows[t][0] = ((t >> 0) & 1) ? -1 : 1;
    for (int i = 1; i < m; ++i) rows[t][i] = ((t >> (1 + coset[i])) & 1) ? -1 : 1;
  }
  // periodic autocorrelation at one shift per coset
  std::vector<std::vector<int>> paf(ncand, std::vector<int>(ncos));
  for (int t = 0; t < ncand; ++t)
    for (int j = 0; j < ncos; ++j) {
      const int s = powmod(g, j, m);
      int acc = 0;
      for (int i = 0; i < m; ++i) acc += rows[t][i] * rows[t][(i + s) % m];
      paf[t][j] = acc;
    }
  std::map<std::vector<int>, std::vector<std::pair<int, int>>> by_sum;
  for (int c = 0; c < ncand; ++c)
    for (int d = c; d < ncand; ++d) {
      std::vector<int> key(ncos);
      for (int j = 0; j < ncos; ++j) key[j] = paf[c][j] + paf[d][j];
      by_sum[key].push_back({c, d});
    }
  int found[4] = {-1, -1, -1, -1};
  for (int a = 0; a < ncand && found[0] < 0; ++a)
    for (int b = a; b < ncand && found[0] < 0; ++b) {
      std::vector<int> key(ncos);
      for (int j = 0; j < ncos; ++j) key[j] = -(paf[a][j] + paf[b][j]);
      auto it = by_sum.find(key);
      if (it == by_sum.end()) continue;
      for (const auto& cd : it->second)  // pairs are stored in lexicographic order
        if (cd.first >= b) {
          found[0] = a, found[1] = b, found[2] = cd.first, found[3] = cd.second;
          break;
        }
    }
  if (found[0] < 0) return {};
  const int n = 4 * m;
  // block (R, C) of the array is sign[R][C] * circulant(which[R][C])
  static const int which[4][4] = {{0, 1, 2, 3}, {1, 0, 3, 2}, {2, 3, 0, 1}, {3, 2, 1, 0}};
  static const int sign[4][4] = {{1, 1, 1, 1}, {-1, 1, -1, 1}, {-1, 1, 1, -1}, {-1, -1, 1, 1}};
  std::vector<int8_t> h(n * n);
  for (int R = 0; R < 4; ++R)
    for (int C = 0; C < 4; ++C) {
      const std::vector<int>& r = rows[found[which[R][C]]];
      for (int i = 0; i < m; ++i)
        for (int j = 0; j < m; ++j)
          h[(R * m + i) * n + (C * m + j)] = static_cast<int8_t>(sign[R][C] * r[((j - i) % m + m) % m]);
    }
  return h;
}

bool is_hadamard(const std::vector<int8_t>& h, int n) {
  for (int i = 0; i < n; ++i)
    for (int j = i; j < n; ++j) {
      int dot = 0;
      for (int k = 0; k < n; ++k) dot += h[i * n + k] * h[j * n + k];
      if (dot != (i == j ? n : 0)) return false;
    }
  return true;
}

}  // namespace

bool hadamard_factor(int n, std::vector<int8_t>* out) {
  std::vector<int8_t> h;
  if (n == 1) {
    h = {1};
  } else if (n == 28) {
    h = paley2(13);
  } else if (n == 172) {
    h = williamson(43, 6);
  } else {
    return false;
  }
  if (h.size() != static_cast<size_t>(n) * n || !is_hadamard(h, n)) return false;
  *out = std::move(h);
  return true;
}

}  // namespace sq
