// Build-time generator: writes the register-resident contraction cores of the
// tensor product for every supported (lmax, parity mode) as straight-line HIP
// device code, from the sparse combined coupling table of cg_builder.
//
// Every coefficient becomes an fp32 literal and every register index a
// compile-time constant, so the per-lane operands stay in VGPRs and the
// coupling table costs no memory traffic at all.  The generated cores are
//   fwd: out[k]  = sum_p W(p) sum_{(i,j,k) in p} C q_ij,  q_ij = x[i] env[j]
//        (products shared by all paths with the same input blocks (a, b))
//   bwd: Q_ij    = sum_{p with blocks (a,b)} sum_k C (W(p) g[k])
//        gx[i]   = sum_j Q_ij env[j]           (overwritten; may alias x)
//        ge[j]  += sum_i Q_ij x[i]             (accumulated across edges)
//   wgrad: acc[p] += sum_k g[k] sum_{(i,j,k) in p} C q_ij
//        (the path-weight gradient of one edge and channel, accumulated)
// which is the tensor product and its VJP with respect to x, env and the path
// weights, written per pair of input blocks so that at most one block of
// temporaries is live.
// W is any accessor with W(p) = the lane's weight of path p.
//
// Usage: gen_kernels <output.inc>
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <stdexcept>
#include <map>
#include <set>
#include <string>
#include <utility>
#include <vector>

#include "cg_builder.hpp"

namespace {

std::string lit(double v) {
  char buf[64];
  std::snprintf(buf, sizeof buf, "%af", double(float(v)));
  return buf;
}

struct Group {  // all paths that share the input blocks (a, b)
  int a, b;
  std::vector<int> paths;
};

std::vector<Group> groups_of(const allegro::TPTable &t) {
  std::vector<Group> gs;
  for (int p = 0; p < int(t.paths.size()); ++p) {
    const auto &ph = t.paths[p];
    if (gs.empty() || gs.back().a != ph.a || gs.back().b != ph.b) gs.push_back({ph.a, ph.b, {}});
    gs.back().paths.push_back(p);
  }
  return gs;
}

// "acc = acc + c * term" with the first assignment and +-1 coefficients folded.
std::string accumulate(const std::string &acc, bool first, double c, const std::string &term) {
  const float cf = float(c);
  if (first) {
    if (cf == 1.0f) return acc + " = " + term + ";";
    if (cf == -1.0f) return acc + " = -" + term + ";";
    return acc + " = " + lit(c) + " * " + term + ";";
  }
  if (cf == 1.0f) return acc + " = " + acc + " + " + term + ";";
  if (cf == -1.0f) return acc + " = " + acc + " - " + term + ";";
  return acc + " = __builtin_fmaf(" + lit(c) + ", " + term + ", " + acc + ");";
}

void emit_core(FILE *f, const allegro::TPTable &t) {
  const int np = int(t.paths.size());
  std::fprintf(f, "template <> struct TPCore<%d, %s> {\n", t.lmax, t.full_parity ? "true" : "false");
  std::fprintf(f, "  static constexpr int LMAX = %d, D1 = %d, D2 = %d, NP = %d, NNZ = %d;\n", t.lmax, t.d1, t.d2, np,
               int(t.entries.size()));
  std::fprintf(f, "  static constexpr bool FULL = %s;\n", t.full_parity ? "true" : "false");
  // x irrep of each component (the per-irrep channel mixing acts block by block)
  std::fprintf(f, "  static constexpr int NX = %d;\n  static constexpr int XIRREP[%d] = {", int(t.x_irreps.size()), t.d1);
  for (int a = 0, k = 0; a < int(t.x_irreps.size()); ++a)
    for (int m = 0; m < 2 * t.x_irreps[a].l + 1; ++m, ++k) std::fprintf(f, "%s%d", k ? ", " : "", a);
  std::fprintf(f, "};\n");

  // entries grouped per path
  std::vector<std::vector<allegro::CGEntry>> per_path(np);
  for (const auto &e : t.entries) per_path[e.path].push_back(e);
  const auto groups = groups_of(t);

  // ---------------------------------------------------------------- forward
  std::fprintf(f,
               "  template <class WT>\n"
               "  static __device__ __forceinline__ void fwd(const float *__restrict__ x, const float *__restrict__ env,\n"
               "                                             const WT &W, float *__restrict__ out) {\n");
  std::vector<bool> out_init(t.d1, false);
  for (const Group &g : groups) {
    std::fprintf(f, "    { // x block %d (l=%d) with env block %d (l=%d)\n", g.a, t.x_irreps[g.a].l, g.b,
                 t.env_irreps[g.b].l);
    std::set<std::pair<int, int>> pairs;
    for (int p : g.paths)
      for (const auto &e : per_path[p]) pairs.insert({e.i, e.j});
    for (const auto &ij : pairs)
      std::fprintf(f, "      const float q%d_%d = x[%d] * env[%d];\n", ij.first, ij.second, ij.first, ij.second);
    for (int p : g.paths) {
      std::map<int, std::vector<allegro::CGEntry>> by_k;
      for (const auto &e : per_path[p]) by_k[e.k].push_back(e);
      for (const auto &kv : by_k) {
        std::fprintf(f, "      { float s;");
        bool first = true;
        for (const auto &e : kv.second) {
          std::fprintf(f, " %s", accumulate("s", first, e.value, "q" + std::to_string(e.i) + "_" + std::to_string(e.j)).c_str());
          first = false;
        }
        const int k = kv.first;
        if (out_init[k])
          std::fprintf(f, " out[%d] = __builtin_fmaf(W(%d), s, out[%d]); }\n", k, p, k);
        else
          std::fprintf(f, " out[%d] = W(%d) * s; }\n", k, p);
        out_init[k] = true;
      }
    }
    std::fprintf(f, "    }\n");
  }
  for (int k = 0; k < t.d1; ++k)
    if (!out_init[k]) std::fprintf(f, "    out[%d] = 0.0f;\n", k);
  std::fprintf(f, "  }\n");

  // ------------------------------------------------- path-weight gradient
  std::fprintf(f,
               "  static __device__ __forceinline__ void wgrad(const float *__restrict__ x, const float *__restrict__ env,\n"
               "                                               const float *__restrict__ g, float (&acc)[NP]) {\n");
  for (const Group &g : groups) {
    std::fprintf(f, "    { // x block %d with env block %d\n", g.a, g.b);
    std::set<std::pair<int, int>> pairs;
    for (int p : g.paths)
      for (const auto &e : per_path[p]) pairs.insert({e.i, e.j});
    for (const auto &ij : pairs)
      std::fprintf(f, "      const float q%d_%d = x[%d] * env[%d];\n", ij.first, ij.second, ij.first, ij.second);
    for (int p : g.paths) {
      std::map<int, std::vector<allegro::CGEntry>> by_k;
      for (const auto &e : per_path[p]) by_k[e.k].push_back(e);
      for (const auto &kv : by_k) {
        std::fprintf(f, "      { float s;");
        bool first = true;
        for (const auto &e : kv.second) {
          std::fprintf(f, " %s", accumulate("s", first, e.value, "q" + std::to_string(e.i) + "_" + std::to_string(e.j)).c_str());
          first = false;
        }
        std::fprintf(f, " acc[%d] = __builtin_fmaf(g[%d], s, acc[%d]); }\n", p, kv.first, p);
      }
    }
    std::fprintf(f, "    }\n");
  }
  std::fprintf(f, "  }\n");

  // ---------------------------------------------------------------- backward
  // Emitted per x irrep a: its x values are read once at the start of the
  // section and its grad_x values are written once at the end, so x and gx may
  // be the same row (in-place) and only one block of gx accumulators is live.
  const int nx = int(t.x_irreps.size());
  std::fprintf(f,
               "  template <class WT>\n"
               "  static __device__ __forceinline__ void bwd(const float *x, const float *__restrict__ env,\n"
               "                                             const WT &W, const float *__restrict__ g,\n"
               "                                             float *gx, float *__restrict__ ge) {\n");
  for (int a = 0; a < nx; ++a) {
    const int la = t.x_irreps[a].l, oa = t.x_off[a], da = 2 * la + 1;
    std::fprintf(f, "    { // x block %d (l=%d)\n", a, la);
    for (int m = 0; m < da; ++m) std::fprintf(f, "      const float xa%d = x[%d];\n", m, oa + m);
    std::vector<bool> gx_init(da, false);
    std::fprintf(f, "      float");
    for (int m = 0; m < da; ++m) std::fprintf(f, "%s gxa%d", m ? "," : "", m);
    std::fprintf(f, ";\n");
    for (const Group &g : groups) {
      if (g.a != a) continue;
      std::fprintf(f, "      { // with env block %d\n", g.b);
      std::set<std::pair<int, int>> wg_needed;  // (path, k)
      for (int p : g.paths)
        for (const auto &e : per_path[p]) wg_needed.insert({p, e.k});
      for (const auto &pk : wg_needed)
        std::fprintf(f, "        const float wg%d_%d = W(%d) * g[%d];\n", pk.first, pk.second, pk.first, pk.second);
      // Q one row i at a time: Q_ij = sum_{p,k} C_ijk wg_pk, then grad_x[i] and
      // the env-gradient terms of that row, so only one row of Q is live.
      std::map<int, std::map<int, std::vector<allegro::CGEntry>>> rows;  // i -> j -> entries
      for (int p : g.paths)
        for (const auto &e : per_path[p]) rows[e.i][e.j].push_back(e);
      for (const auto &row : rows) {
        const int i = row.first, m = i - oa;
        std::fprintf(f, "        {\n");
        for (const auto &cell : row.second) {
          const int j = cell.first;
          const std::string name = "Q" + std::to_string(i) + "_" + std::to_string(j);
          bool first = true;
          for (const auto &e : cell.second) {
            std::fprintf(f, "          %s%s\n", first ? "float " : "",
                         accumulate(name, first, e.value, "wg" + std::to_string(e.path) + "_" + std::to_string(e.k)).c_str());
            first = false;
          }
        }
        for (const auto &cell : row.second) {
          const int j = cell.first;
          if (gx_init[m])
            std::fprintf(f, "          gxa%d = __builtin_fmaf(Q%d_%d, env[%d], gxa%d);", m, i, j, j, m);
          else
            std::fprintf(f, "          gxa%d = Q%d_%d * env[%d];", m, i, j, j);
          gx_init[m] = true;
          std::fprintf(f, " ge[%d] = __builtin_fmaf(Q%d_%d, xa%d, ge[%d]);\n", j, i, j, m, j);
        }
        std::fprintf(f, "        }\n");
      }
      std::fprintf(f, "      }\n");
    }
    for (int m = 0; m < da; ++m)
      std::fprintf(f, "      gx[%d] = %s;\n", oa + m, gx_init[m] ? ("gxa" + std::to_string(m)).c_str() : "0.0f");
    std::fprintf(f, "    }\n");
  }
  std::fprintf(f, "  }\n};\n\n");
}

// The forward as a per-center matrix: out[k] = sum_i M[k][i] x[i] with
//   M[k][i] = sum_{p = (a(i), b, c(k))} W(p) sum_j C_pijk env[j],
// which depends only on the center and the channel.  Its rows are split over
// NW waves (ROWS consecutive rows each); wave w builds its rows once per
// center and applies them to every edge.  Emitted for lmax 3, where it takes
// about half the arithmetic of the direct contraction per edge.
void emit_matrix(FILE *f, const allegro::TPTable &t, int nw, const char *name) {
  const int d1 = t.d1, rows = d1 / nw;
  // (row k, column i) -> list of (path, j, C)
  std::map<std::pair<int, int>, std::vector<allegro::CGEntry>> cells;
  for (const auto &e : t.entries) cells[{e.k, e.i}].push_back(e);
  int maxm = 0;
  std::vector<std::vector<std::pair<int, int>>> wave_cells(nw);
  for (int w = 0; w < nw; ++w) {
    for (const auto &kv : cells)
      if (kv.first.first / rows == w) wave_cells[w].push_back(kv.first);
    maxm = std::max(maxm, int(wave_cells[w].size()));
  }
  std::fprintf(f, "template <> struct %s<%d, %s> {\n", name, t.lmax, t.full_parity ? "true" : "false");
  std::fprintf(f, "  static constexpr int NW = %d, ROWS = %d, MAXM = %d;\n", nw, rows, maxm);
  // build
  std::fprintf(f, "  template <class WT>\n  static __device__ __forceinline__ void build(int w, const float *__restrict__ env, "
                  "const WT &W, float (&m)[MAXM]) {\n    switch (w) {\n");
  for (int w = 0; w < nw; ++w) {
    std::fprintf(f, "      case %d: {\n", w);
    for (int q = 0; q < int(wave_cells[w].size()); ++q) {
      const auto &es = cells[wave_cells[w][q]];
      std::map<int, std::vector<allegro::CGEntry>> by_path;
      for (const auto &e : es) by_path[e.path].push_back(e);
      std::fprintf(f, "        {");
      bool first_p = true;
      for (const auto &pv : by_path) {
        std::fprintf(f, " { float s;");
        bool first = true;
        for (const auto &e : pv.second) {
          std::fprintf(f, " %s", accumulate("s", first, e.value, "env[" + std::to_string(e.j) + "]").c_str());
          first = false;
        }
        if (first_p)
          std::fprintf(f, " m[%d] = W(%d) * s; }", q, pv.first);
        else
          std::fprintf(f, " m[%d] = __builtin_fmaf(W(%d), s, m[%d]); }", q, pv.first, q);
        first_p = false;
      }
      std::fprintf(f, " }\n");
    }
    for (int q = int(wave_cells[w].size()); q < maxm; ++q) std::fprintf(f, "        m[%d] = 0.0f;\n", q);
    std::fprintf(f, "      } break;\n");
  }
  std::fprintf(f, "      default: break;\n    }\n  }\n");
  // apply: one FMA chain per row of the wave, over the lane's x row in registers
  std::fprintf(f, "  static __device__ __forceinline__ void apply(int w, const float (&x)[%d], const float (&m)[MAXM], "
                  "float (&o)[ROWS]) {\n    switch (w) {\n", d1);
  for (int w = 0; w < nw; ++w) {
    std::fprintf(f, "      case %d:\n", w);
    for (int r = 0; r < rows; ++r) {
      const int k = w * rows + r;
      std::fprintf(f, "        o[%d] =", r);
      bool first = true;
      std::string expr;
      for (int q = 0; q < int(wave_cells[w].size()); ++q) {
        if (wave_cells[w][q].first != k) continue;
        const int i = wave_cells[w][q].second;
        const std::string term = "m[" + std::to_string(q) + "], x[" + std::to_string(i) + "]";
        expr = first ? "m[" + std::to_string(q) + "] * x[" + std::to_string(i) + "]"
                     : "__builtin_fmaf(" + term + ", " + expr + ")";
        first = false;
      }
      std::fprintf(f, " %s;\n", first ? "0.0f" : expr.c_str());
    }
    std::fprintf(f, "        break;\n");
  }
  std::fprintf(f, "      default: break;\n    }\n  }\n};\n\n");
}

// Lane tables of the matrix-core backward at lmax 3 (tp_mfma_bwd_kernel).
//
// Per (center, channel) the backward needs two small dense products:
//   grad_x[e][i] = sum_k g[e][k] M[k][i]      (M the per-center matrix of the forward)
//   G[k][i]      = sum_e g[e][k] x[e][i]      (per-center products)
// which run on v_mfma_f32_16x16x4f32.  In its operand and result layout lane
// l = 16 h + c of a wave holds, for slot s = (tk * NT + ti) * 4 + r, the cell
//   (k, i) = (16 tk + 4 h + r, 16 ti + c)
// of M (as the A operand of grad_x^T = M^T g^T, K = k), and the same cell of G
// (the accumulator) except with d1 = 32, where G's operands are read as pairs
// of adjacent columns and the lane holds G's cell (2 (4 h + r) + tk, 2 c + ti).
// M and G cross between waves as a lane-major spill (spill_pos).  The tables let every lane
// form its own cells of M and contract its cells of G without any lane-uniform
// code:
//   Z[q] = W(p) env[j] for the q-th distinct (p, j) of the coupling table
//          (rounds of 64 lanes; word p | j << 16 per lane);
//   M[s] = sum_t MC[t][s][lane] Z[MI[t][s][lane]]   (at most MT terms per cell,
//          padded with zero coefficients);
//   H[q] = sum over the cells (k, i) of path p, env component j of C_pijk G[k][i]
//          (H rounds: lane -> target q, HT[round] terms of (coefficient, index
//          of the cell in the G spill));
//   grad_env[j] = sum_q W(p(q)) H[q] over the q with j(q) = j: lane 4 j + quarter
//          sums every fourth such q (words q | p << 16, padded with q = NZ,
//          where H[NZ] = 0), then the four quarters are added by lane shuffles;
//   grad_W[p]   = sum over the q of path p (contiguous from off, len of them) of
//          env[j(q)] H[q] (word off | len << 16).
// All tables are packed into one array of 32-bit words (floats as their bit
// patterns, 16-bit indices two per word), copied to LDS once per workgroup.
void emit_mfma_tables(FILE *f, const allegro::TPTable &t) {
  const int d1 = t.d1, np = int(t.paths.size()), nt = d1 / 16, S = nt * nt * 4;
  if (d1 % 16 != 0 || t.d2 != 16) throw std::runtime_error("matrix-core tables need d1 % 16 == 0 and d2 == 16");
  // distinct (p, j), sorted
  std::map<std::pair<int, int>, int> zq;
  for (const auto &e : t.entries) zq[{e.path, e.j}] = 0;
  std::vector<std::pair<int, int>> zlist;
  for (auto &kv : zq) {
    kv.second = int(zlist.size());
    zlist.push_back(kv.first);
  }
  const int nz = int(zlist.size()), rz = (nz + 63) / 64;
  auto cell_of = [&](int lane, int slot) {
    const int h = lane / 16, c = lane % 16, r = slot % 4, tk = (slot / 4) / nt, ti = (slot / 4) % nt;
    return std::make_pair(16 * tk + 4 * h + r, 16 * ti + c);  // (k, i)
  };
  // With d1 = 32 the kernel reads the G products' operands as pairs of adjacent
  // columns, so product tile t (of the two per operand) takes the columns 2 c + t
  // and G's cell (k, i) sits in tile (k % 2, i % 2) at row k / 2, column i / 2.
  // The spill of a lane's cells is lane-major: the S slots of lane l start at
  // l S, in groups of four (one 16-byte access) whose order is XOR-swizzled by
  // (l / 4) mod (S / 4), so that eight lanes' 16-byte accesses hit distinct banks.
  const bool gpair = d1 == 32;
  auto spill_pos = [&](int lane, int slot) {
    const int q = slot / 4, r = slot % 4;
    return lane * S + 4 * (q ^ ((lane / 4) & (S / 4 - 1))) + r;
  };
  auto gidx_of = [&](int k, int i) {  // position of cell (k, i) in the spill
    if (gpair) {
      const int tk = k % 2, m = k / 2, h = m / 4, r = m % 4, ti = i % 2, c = i / 2;
      return spill_pos(16 * h + c, (tk * nt + ti) * 4 + r);
    }
    const int tk = k / 16, h = (k % 16) / 4, r = k % 4, ti = i / 16, c = i % 16;
    return spill_pos(16 * h + c, (tk * nt + ti) * 4 + r);
  };
  // M terms per cell
  std::map<std::pair<int, int>, std::vector<std::pair<double, int>>> mterms;
  for (const auto &e : t.entries) mterms[{e.k, e.i}].push_back({e.value, zq[{e.path, e.j}]});
  int mt = 0;
  for (const auto &kv : mterms) mt = std::max(mt, int(kv.second.size()));
  // H terms per (p, j); rounds by descending term count
  std::vector<std::vector<std::pair<double, int>>> hterms(nz);
  for (const auto &e : t.entries) hterms[zq[{e.path, e.j}]].push_back({e.value, gidx_of(e.k, e.i)});
  std::vector<int> order(nz);
  for (int q = 0; q < nz; ++q) order[q] = q;
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return hterms[a].size() > hterms[b].size(); });
  const int rh = (nz + 63) / 64;
  std::vector<int> ht(rh, 0);
  for (int k = 0; k < nz; ++k) ht[k / 64] = std::max(ht[k / 64], int(hterms[order[k]].size()));
  int th = 0;
  for (int v : ht) th += v;
  // grad_env lists: lane 4 j + quarter
  std::vector<std::vector<int>> ge_lane(64);
  for (int j = 0; j < 16; ++j) {
    std::vector<int> qs;
    for (int q = 0; q < nz; ++q)
      if (zlist[q].second == j) qs.push_back(q);
    for (size_t n = 0; n < qs.size(); ++n) ge_lane[4 * j + int(n % 4)].push_back(qs[n]);
  }
  int tge = 0;
  for (const auto &v : ge_lane) tge = std::max(tge, int(v.size()));
  const int rpw = (np + 63) / 64;
  // pack
  std::vector<uint32_t> words;
  auto fbits = [](double v) {
    const float x = float(v);
    uint32_t u;
    std::memcpy(&u, &x, 4);
    return u;
  };
  auto push16 = [&](const std::vector<int> &v) {  // 64 indices -> 32 words
    for (int l = 0; l < 64; l += 2) words.push_back(uint32_t(v[l]) | (uint32_t(v[l + 1]) << 16));
  };
  const int off_mc = int(words.size());
  for (int tt = 0; tt < mt; ++tt)
    for (int sl = 0; sl < S; ++sl)
      for (int l = 0; l < 64; ++l) {
        const auto &v = mterms[cell_of(l, sl)];
        words.push_back(fbits(tt < int(v.size()) ? v[tt].first : 0.0));
      }
  const int off_zp = int(words.size());
  for (int q = 0; q < rz * 64; ++q)
    words.push_back(q < nz ? uint32_t(zlist[q].first) | (uint32_t(zlist[q].second) << 16) : 0u);
  const int off_hc = int(words.size());
  for (int r = 0; r < rh; ++r)
    for (int tt = 0; tt < ht[r]; ++tt)
      for (int l = 0; l < 64; ++l) {
        const int k = 64 * r + l;
        const bool ok = k < nz && tt < int(hterms[order[k]].size());
        words.push_back(fbits(ok ? hterms[order[k]][tt].first : 0.0));
      }
  const int off_ge = int(words.size());
  for (int tt = 0; tt < tge; ++tt)
    for (int l = 0; l < 64; ++l) {
      const int q = tt < int(ge_lane[l].size()) ? ge_lane[l][tt] : nz;
      const int pth = q < nz ? zlist[q].first : 0;
      words.push_back(uint32_t(q) | (uint32_t(pth) << 16));
    }
  const int off_pw = int(words.size());
  int pwmax = 0;
  for (int p = 0; p < rpw * 64; ++p) {
    int off = 0, len = 0;
    for (int q = 0; q < nz; ++q)
      if (zlist[q].first == p) {
        if (!len) off = q;
        if (q != off + len) throw std::runtime_error("the (p, j) list of a path is not contiguous");
        ++len;
      }
    pwmax = std::max(pwmax, len);
    words.push_back(uint32_t(off) | (uint32_t(len) << 16));
  }
  const int off_mi = int(words.size());
  for (int tt = 0; tt < mt; ++tt)
    for (int sl = 0; sl < S; ++sl) {
      std::vector<int> v(64);
      for (int l = 0; l < 64; ++l) {
        const auto &m = mterms[cell_of(l, sl)];
        v[l] = tt < int(m.size()) ? m[tt].second : 0;
      }
      push16(v);
    }
  const int off_hi = int(words.size());
  for (int r = 0; r < rh; ++r)
    for (int tt = 0; tt < ht[r]; ++tt) {
      std::vector<int> v(64);
      for (int l = 0; l < 64; ++l) {
        const int k = 64 * r + l;
        v[l] = (k < nz && tt < int(hterms[order[k]].size())) ? hterms[order[k]][tt].second : 0;
      }
      push16(v);
    }
  const int off_ht = int(words.size());
  for (int r = 0; r < rh; ++r) {
    std::vector<int> v(64);
    for (int l = 0; l < 64; ++l) v[l] = 64 * r + l < nz ? order[64 * r + l] : nz + 1;
    push16(v);
  }
  while (words.size() % 4) words.push_back(0u);
  const char *full = t.full_parity ? "true" : "false";
  std::fprintf(f, "template <> struct TPMfmaTab<%d, %s> {\n", t.lmax, full);
  std::fprintf(f, "  static constexpr int D1 = %d, NT = %d, S = %d, NP = %d, NZ = %d, RZ = %d, MT = %d, RH = %d, TH = %d, "
                  "TGE = %d, RPW = %d, PWMAX = %d;\n", d1, nt, S, np, nz, rz, mt, rh, th, tge, rpw, pwmax);
  std::fprintf(f, "  static constexpr bool GPAIR = %s;  // G operands read as column pairs\n", gpair ? "true" : "false");
  std::fprintf(f, "  static constexpr int HT[%d] = {", rh);
  for (int r = 0; r < rh; ++r) std::fprintf(f, "%s%d", r ? ", " : "", ht[r]);
  std::fprintf(f, "};\n");
  std::fprintf(f, "  static constexpr int OFF_MC = %d, OFF_ZP = %d, OFF_HC = %d, OFF_GE = %d, OFF_PW = %d, OFF_MI = %d, "
                  "OFF_HI = %d, OFF_HT = %d, WORDS = %d;\n", off_mc, off_zp, off_hc, off_ge, off_pw, off_mi, off_hi,
               off_ht, int(words.size()));
  std::fprintf(f, "  static __device__ const uint32_t *words();\n};\n");
  std::fprintf(f, "static __device__ __attribute__((aligned(16))) const uint32_t kMfmaTab%d%s[%d] = {", t.lmax,
               t.full_parity ? "F" : "N", int(words.size()));
  for (size_t q = 0; q < words.size(); ++q)
    std::fprintf(f, "%s0x%08x", q == 0 ? "\n  " : (q % 8 ? ", " : ",\n  "), words[q]);
  std::fprintf(f, "};\n");
  std::fprintf(f, "__device__ inline const uint32_t *TPMfmaTab<%d, %s>::words() { return kMfmaTab%d%s; }\n\n", t.lmax,
               full, t.lmax, t.full_parity ? "F" : "N");
}

}  // namespace

int main(int argc, char **argv) {
  if (argc != 2) {
    std::fprintf(stderr, "usage: %s <output.inc>\n", argv[0]);
    return 2;
  }
  FILE *f = std::fopen(argv[1], "w");
  if (!f) {
    std::perror(argv[1]);
    return 1;
  }
  std::fprintf(f,
               "// Generated by gen_kernels from the sparse coupling table of cg_builder. Do not edit.\n"
               "#pragma once\n\n"
               "template <int LMAX, bool FULL> struct TPCore;\n"
               "template <int LMAX, bool FULL> struct TPMFwd;\n"

               "template <int LMAX, bool FULL> struct TPMfmaTab;\n\n");
  try {
    for (int lmax = 1; lmax <= 3; ++lmax)
      for (int full = 0; full <= 1; ++full) emit_core(f, allegro::build_table(lmax, full != 0));
    for (int full = 0; full <= 1; ++full) {
      const allegro::TPTable t3 = allegro::build_table(3, full != 0);
      emit_matrix(f, t3, 8, "TPMFwd");
      emit_mfma_tables(f, t3);
    }
  } catch (const std::exception &ex) {
    std::fprintf(stderr, "gen_kernels: %s\n", ex.what());
    std::fclose(f);
    return 1;
  }
  std::fclose(f);
  return 0;
}
