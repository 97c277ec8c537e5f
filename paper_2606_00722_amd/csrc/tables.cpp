// Host-side constant tables of the HIP path.
//
// Everything here depends only on the lexer, the grammar and the vocabulary,
// never on a sequence; it is computed once when a context is created.
//
//  * Dotted items, numbered consecutively per production so that advancing
//    the dot is a one-bit left shift of an item bitset; the augmented
//    production S' -> S comes last.  Prediction tables use the left-corner
//    closure (Alg. 3's predict step applied until nothing new appears;
//    nullable prefixes are left to completion at run time).
//  * The lexer's gap automaton.  A masked run reads Sigma* (Limitations), so
//    inside it a lexeme extends along any byte, and a lexeme ends on a byte
//    that cannot extend it but starts a new one.  The lexeme-level nodes of a
//    gap are the "fresh" states delta(q0, c) reached right after an emission.
//    Fresh states with the same left language for every state in which the
//    gap can be entered are merged (exactly: their membership in every subset
//    of the gap automaton's determinisation, over all entry states, agrees).
//    Merging nodes with equal left languages keeps the language of the
//    completion automaton, so Valid is unchanged.  For lexers where whitespace
//    can separate any two lexemes this leaves two classes per gap.
//  * The regular cover of App. A.2: its rule-position states are the dotted
//    items; entry/exit states of each nonterminal are extra bits.
#include "tables.h"

#include <algorithm>
#include <functional>
#include <map>
#include <set>
#include <vector>

#include "../../include/epic.h"

namespace epic {
namespace {

struct Bits {
  std::vector<uint64_t> w;
  explicit Bits(int n = 0) : w((n + 63) / 64, 0) {}
  void set(int i) { w[i >> 6] |= 1ull << (i & 63); }
  bool get(int i) const { return (w[i >> 6] >> (i & 63)) & 1; }
  bool any() const {
    for (uint64_t x : w)
      if (x) return true;
    return false;
  }
  bool operator<(const Bits& o) const { return w < o.w; }
  bool operator==(const Bits& o) const { return w == o.w; }
};

inline void set32(std::vector<uint32_t>& v, size_t base, int i) { v[base + (i >> 5)] |= 1u << (i & 31); }

// Terminal strings of the derivations inside a masked run (witness
// extraction).  Nonterminal derivations between classes are found in rounds
// (a derivation found in round r uses terminal edges, epsilon paths and
// derivations of earlier rounds only), so expanding one terminates; the
// strings are the expansions.  Item prefixes of a run's own entries follow a
// breadth-first search over (class, item) from the start items at class j.
void build_witness_strings(HostTables& H, int K, const std::vector<char>& epsp, int T, int N, int P,
                           const int32_t* lhs, const int32_t* roff, const int32_t* rhs, const std::vector<int>& base) {
  const int NI = H.NI, KK = std::max(K, 1), W = H.W;
  constexpr size_t kPoolCap = (size_t)8 << 20;
  H.wy_nt.assign((size_t)KK * KK * N, -1);
  H.wy_own.assign((size_t)KK * KK * NI, -1);
  H.wy_pool.clear();
  if (K == 0) return;
  struct Deriv {
    int round = 0, prod = -1;
    std::vector<int> cls;   // class after each symbol (cls[0]: after the leading epsilon path)
    std::vector<int> via;   // terminal symbol i: the class its edge leaves from
  };
  std::vector<Deriv> der((size_t)K * K * N);
  auto at = [&](int A, int j, int k) -> Deriv& { return der[((size_t)j * K + k) * N + A]; };
  for (int round = 1;; ++round) {
    std::vector<std::pair<size_t, Deriv>> found;
    for (int p = 0; p < P; ++p) {
      const int A = lhs[p] - T, m = roff[p + 1] - roff[p];
      for (int j = 0; j < K; ++j) {
        // pred[i][c]: class before symbol i reaching class c after it (-1: unreached);
        // from[i][c]: for terminal symbols, the class the edge leaves from
        std::vector<std::vector<int>> pred(m + 1, std::vector<int>(K, -1)), from(m + 1, std::vector<int>(K, -1));
        for (int c = 0; c < K; ++c)
          if (epsp[(size_t)j * K + c]) pred[0][c] = j;
        for (int i = 1; i <= m; ++i) {
          const int X = rhs[roff[p] + i - 1];
          for (int c = 0; c < K; ++c) {
            if (pred[i - 1][c] < 0) continue;
            for (int c2 = 0; c2 < K; ++c2) {
              if (X < T) {
                if (!((H.cls_internal[(size_t)c * K + c2] >> X) & 1)) continue;
                for (int c3 = 0; c3 < K; ++c3)
                  if (epsp[(size_t)c2 * K + c3] && pred[i][c3] < 0) {
                    pred[i][c3] = c;
                    from[i][c3] = c2;
                  }
              } else {
                const Deriv& d = at(X - T, c, c2);
                if (d.prod >= 0 && d.round < round && pred[i][c2] < 0) pred[i][c2] = c;
              }
            }
          }
        }
        for (int k = 0; k < K; ++k) {
          if (pred[m][k] < 0 || at(A, j, k).prod >= 0) continue;
          Deriv d;
          d.round = round;
          d.prod = p;
          d.cls.assign(m + 1, 0);
          d.via.assign(m + 1, -1);
          int c = k;
          for (int i = m; i >= 1; --i) {
            d.cls[i] = c;
            d.via[i] = from[i][c];
            c = pred[i][c];
          }
          d.cls[0] = c;
          found.push_back({((size_t)j * K + k) * N + A, d});
        }
      }
    }
    int added = 0;
    for (auto& f : found)
      if (der[f.first].prod < 0) {
        der[f.first] = f.second;
        ++added;
      }
    if (!added) break;
  }
  // expansions, memoised per (A, j, k)
  std::vector<std::vector<uint8_t>> str((size_t)K * K * N);
  std::vector<char> done((size_t)K * K * N, 0);
  bool overflow = false;
  std::function<const std::vector<uint8_t>&(int, int, int)> expand = [&](int A, int j, int k) -> const std::vector<uint8_t>& {
    const size_t id = ((size_t)j * K + k) * N + A;
    if (done[id]) return str[id];
    const Deriv& d = der[id];
    std::vector<uint8_t> out;
    const int m = roff[d.prod + 1] - roff[d.prod];
    for (int i = 1; i <= m && !overflow; ++i) {
      const int X = rhs[roff[d.prod] + i - 1];
      if (X < T) {
        out.push_back((uint8_t)X);
      } else {
        const std::vector<uint8_t>& sub = expand(X - T, d.cls[i - 1], d.cls[i]);
        out.insert(out.end(), sub.begin(), sub.end());
      }
      if (out.size() > 4096) overflow = true;
    }
    done[id] = 1;
    str[id] = std::move(out);
    return str[id];
  };
  auto put = [&](const std::vector<uint8_t>& v) -> int32_t {
    if (v.size() > 0xFFFF || H.wy_pool.size() + v.size() + 2 > kPoolCap) return -1;
    const int32_t off = (int32_t)H.wy_pool.size();
    H.wy_pool.push_back((uint8_t)(v.size() & 0xFF));
    H.wy_pool.push_back((uint8_t)(v.size() >> 8));
    H.wy_pool.insert(H.wy_pool.end(), v.begin(), v.end());
    return off;
  };
  for (int j = 0; j < K; ++j)
    for (int k = 0; k < K; ++k)
      for (int A = 0; A < N; ++A)
        if (at(A, j, k).prod >= 0) {
          overflow = false;
          const std::vector<uint8_t>& v = expand(A, j, k);
          if (!overflow) H.wy_nt[((size_t)j * K + k) * N + A] = put(v);
        }
  // item prefixes of a run's own entries: breadth-first over (class, item)
  std::vector<int> prod_of(NI, -1);
  for (int p = 0; p <= P; ++p) {
    const int len = p < P ? roff[p + 1] - roff[p] : 1;
    for (int d = 0; d <= len; ++d) prod_of[base[p] + d] = p;
  }
  for (int j = 0; j < K; ++j) {
    std::vector<int> par((size_t)K * NI, -2);  // parent state, -1 for a start item at class j
    std::vector<std::vector<uint8_t>> pre((size_t)K * NI);
    std::vector<int> queue;
    for (int p = 0; p < P; ++p) {
      const int s = j * NI + base[p];
      par[s] = -1;
      queue.push_back(s);
    }
    for (size_t qi = 0; qi < queue.size(); ++qi) {
      const int s = queue[qi], c = s / NI, it = s % NI;
      auto visit = [&](int c2, int it2, const std::vector<uint8_t>* add) {
        const int s2 = c2 * NI + it2;
        if (par[s2] != -2) return;
        par[s2] = s;
        pre[s2] = pre[s];
        if (add) pre[s2].insert(pre[s2].end(), add->begin(), add->end());
        queue.push_back(s2);
      };
      for (int c2 = 0; c2 < K; ++c2)
        if (c2 != c && epsp[(size_t)c * K + c2]) visit(c2, it, nullptr);
      const int sym = H.next_sym[it];
      if (sym < 0 || prod_of[it] >= P) continue;
      for (int c2 = 0; c2 < K; ++c2) {
        if (sym < 64) {
          if ((H.cls_internal[(size_t)c * K + c2] >> sym) & 1) {
            const std::vector<uint8_t> t{(uint8_t)sym};
            visit(c2, it + 1, &t);
          }
        } else {
          const int32_t off = H.wy_nt[((size_t)c * K + c2) * N + (sym - 64)];
          if (off >= 0) {
            const int len = H.wy_pool[off] | (H.wy_pool[off + 1] << 8);
            const std::vector<uint8_t> t(H.wy_pool.begin() + off + 2, H.wy_pool.begin() + off + 2 + len);
            visit(c2, it + 1, &t);
          }
        }
      }
    }
    for (int k = 0; k < K; ++k)
      for (int it = 0; it < NI; ++it)
        if (par[(size_t)k * NI + it] != -2 && ((H.gap_own[((size_t)j * K + k) * W + (it >> 5)] >> (it & 31)) & 1))
          H.wy_own[((size_t)j * K + k) * NI + it] = put(pre[(size_t)k * NI + it]);
  }
}

}  // namespace

int build_tables(int Q, const int16_t* trans, const int16_t* accept, int T, int N, int start, int P,
                 const int32_t* lhs, const int32_t* roff, const int32_t* rhs, int V, const uint8_t* vbytes,
                 const int32_t* voffs, HostTables& H, std::string& why) {
  // ---------------------------------------------------------------- checks
  if (T < 1 || T > kMaxTerminals || N < 1 || N > kMaxNonterminals) {
    why = "grammar has too many terminals or nonterminals";
    return EPIC_ERR_UNSUPPORTED;
  }
  if (Q < 1 || Q > kMaxStates) {
    why = "lexer has too many states";
    return EPIC_ERR_UNSUPPORTED;
  }
  if (accept[0] != -1) {
    why = "lexer start state accepts";
    return EPIC_ERR_LEXER;
  }
  for (int q = 0; q < Q; ++q) {
    int a = accept[q];
    if (!(a == -1 || a == -2 || (a >= 0 && a < T))) {
      why = "lexer accept label out of range";
      return EPIC_ERR_LEXER;
    }
    for (int c = 0; c < 256; ++c)
      if (trans[q * 256 + c] < -1 || trans[q * 256 + c] >= Q) {
        why = "lexer transition out of range";
        return EPIC_ERR_LEXER;
      }
  }
  {  // trim: every state reaches an accepting state
    std::vector<char> live(Q, 0);
    for (int q = 0; q < Q; ++q) live[q] = accept[q] != -1;
    bool changed = true;
    while (changed) {
      changed = false;
      for (int q = 0; q < Q; ++q)
        if (!live[q])
          for (int c = 0; c < 256; ++c) {
            int d = trans[q * 256 + c];
            if (d >= 0 && live[d]) {
              live[q] = 1;
              changed = true;
              break;
            }
          }
    }
    for (int q = 0; q < Q; ++q)
      if (!live[q]) {
        why = "lexer DFA is not trim";
        return EPIC_ERR_LEXER;
      }
  }
  if (P < 1 || start < T || start >= T + N || roff[0] != 0) {
    why = "bad grammar header";
    return EPIC_ERR_GRAMMAR;
  }
  for (int p = 0; p < P; ++p) {
    if (lhs[p] < T || lhs[p] >= T + N || roff[p + 1] < roff[p]) {
      why = "bad production";
      return EPIC_ERR_GRAMMAR;
    }
    for (int k = roff[p]; k < roff[p + 1]; ++k)
      if (rhs[k] < 0 || rhs[k] >= T + N) {
        why = "undefined symbol";
        return EPIC_ERR_GRAMMAR;
      }
  }
  if (V < 1) {
    why = "empty vocabulary";
    return EPIC_ERR_VOCAB;
  }
  for (int t = 0; t < V; ++t) {
    int len = voffs[t + 1] - voffs[t];
    if (len < 1 || len > 8) {
      why = "token length must be 1..8 bytes";
      return EPIC_ERR_VOCAB;
    }
  }

  H = HostTables();
  H.Q = Q;
  H.T = T;
  H.N = N;
  H.P = P;
  H.V = V;
  H.QW = (Q + 31) / 32;
  H.trans.assign(trans, trans + (size_t)Q * 256);
  H.accept.assign(accept, accept + Q);
  H.vbytes.assign(vbytes, vbytes + voffs[V]);
  if (H.vbytes.empty()) H.vbytes.push_back(0);
  H.voffs.assign(voffs, voffs + V + 1);

  // ---------------------------------------------------------------- items
  // Dotted items of production p are base[p] .. base[p]+|rhs_p|.  Productions
  // are packed into 32-bit words first-fit by decreasing length, so that no
  // production straddles a word: advancing the dot is then a shift inside
  // one word, and closing an item set over a self-loop of the completion
  // graph is one integer addition per word (the carry runs along a
  // production's consecutive items and stops at its first item that cannot
  // advance).
  std::vector<int> base(P + 1);
  std::vector<int> order(P + 1);
  for (int p = 0; p <= P; ++p) {
    order[p] = p;
    int len = p < P ? roff[p + 1] - roff[p] : 1;
    H.max_rhs = std::max(H.max_rhs, len);
    if (len + 1 > 32) {
      why = "a production has more than 31 symbols";
      return EPIC_ERR_UNSUPPORTED;
    }
  }
  auto plen = [&](int p) { return (p < P ? roff[p + 1] - roff[p] : 1) + 1; };
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return plen(a) > plen(b); });
  std::vector<int> fill;  // items used in each word
  for (int p : order) {
    int need = plen(p), w = 0;
    while (w < (int)fill.size() && fill[w] + need > 32) ++w;
    if (w == (int)fill.size()) fill.push_back(0);
    base[p] = w * 32 + fill[w];
    fill[w] += need;
  }
  int W = 1;
  while (W < (int)fill.size()) W *= 2;
  if (W > kMaxItemWords) {
    why = "more than 512 dotted items";
    return EPIC_ERR_UNSUPPORTED;
  }
  const int ni = W * 32;
  H.NI = ni;
  H.W = W;
  H.CW = W + 4;  // cover state: items, then entry bits (2 words), then exit bits (2 words)
  H.start_nt = start - T;
  H.start_item = base[P];
  H.goal_item = base[P] + 1;
  H.exp_t.assign((size_t)T * W, 0);
  H.exp_n.assign((size_t)N * W, 0);
  H.pred.assign((size_t)N * W, 0);
  H.complete.assign(W, 0);
  H.item_lhs.assign(ni, -1);
  H.next_nt.assign(ni, -1);
  H.next_sym.assign(ni, -1);
  H.start_of.assign((size_t)N * W, 0);
  H.end_of.assign((size_t)N * W, 0);
  for (int p = 0; p <= P; ++p) {
    int len = p < P ? roff[p + 1] - roff[p] : 1;
    int A = p < P ? lhs[p] - T : -1;
    for (int k = 0; k <= len; ++k) {
      int it = base[p] + k;
      H.item_lhs[it] = (int8_t)A;
      if (k < len) {
        int X = p < P ? rhs[roff[p] + k] : start;
        if (X < T) {
          set32(H.exp_t, (size_t)X * W, it);
          H.next_sym[it] = (int8_t)X;
        } else {
          set32(H.exp_n, (size_t)(X - T) * W, it);
          H.next_nt[it] = (int8_t)(X - T);
          H.next_sym[it] = (int8_t)(64 + X - T);
        }
      } else if (p < P) {
        set32(H.complete, 0, it);
      }
    }
    if (p < P) {
      set32(H.start_of, (size_t)A * W, base[p]);
      set32(H.end_of, (size_t)A * W, base[p] + len);
    }
  }
  // nullable nonterminals (derive the empty string)
  uint64_t nullable = 0;
  for (bool changed = true; changed;) {
    changed = false;
    for (int p = 0; p < P; ++p) {
      int A = lhs[p] - T;
      if ((nullable >> A) & 1) continue;
      bool all = true;
      for (int k = roff[p]; k < roff[p + 1] && all; ++k) all = rhs[k] >= T && ((nullable >> (rhs[k] - T)) & 1);
      if (all) {
        nullable |= 1ull << A;
        changed = true;
      }
    }
  }
  H.nullable = nullable;
  // item-set helpers over W words
  typedef std::vector<uint32_t> Set;
  auto exp_mask = [&](uint64_t nts) {
    Set m(W, 0);
    for (int B = 0; B < N; ++B)
      if ((nts >> B) & 1)
        for (int w = 0; w < W; ++w) m[w] |= H.exp_n[(size_t)B * W + w];
    return m;
  };
  auto adv_or = [&](const Set& x, const Set& m, Set& out) {  // out |= (x & m) << 1, true if out grew
    bool grew = false;
    for (int w = 0; w < W; ++w) {
      uint32_t a = (x[w] & m[w]) << 1;
      if (a & ~out[w]) grew = true;
      out[w] |= a;
    }
    return grew;
  };
  H.mn.assign(W, 0);
  {
    Set m = exp_mask(nullable);
    for (int w = 0; w < W; ++w) H.mn[w] = m[w];
  }
  auto nclose = [&](Set& x) {  // advance over nullable nonterminals until nothing changes
    while (adv_or(x, H.mn, x)) {
    }
  };
  // Prediction closure of each nonterminal B: the items A -> . gamma for A
  // predicted from B, closed under skipping nullable nonterminals and under
  // predicting every nonterminal such an item expects (Alg. 3's predict step
  // together with the empty completions of nullable nonterminals).
  for (int B = 0; B < N; ++B) {
    Set x(W, 0);
    uint64_t predicted = 0, todo = 1ull << B;
    while (todo) {
      predicted |= todo;
      for (int A = 0; A < N; ++A)
        if ((todo >> A) & 1)
          for (int w = 0; w < W; ++w) x[w] |= H.start_of[(size_t)A * W + w];
      nclose(x);
      uint64_t e = 0;
      for (int i = 0; i < ni; ++i)
        if (((x[i >> 5] >> (i & 31)) & 1) && H.next_nt[i] >= 0) e |= 1ull << H.next_nt[i];
      todo = e & ~predicted;
    }
    for (int w = 0; w < W; ++w) H.pred[(size_t)B * W + w] = x[w];
  }
  H.expn_nib.assign((size_t)16 * 16 * W, 0);
  H.pred_nib.assign((size_t)16 * 16 * W, 0);
  for (int i = 0; i < 16; ++i)
    for (int v = 0; v < 16; ++v)
      for (int b = 0; b < 4; ++b) {
        const int B = 4 * i + b;
        if (!((v >> b) & 1) || B >= N) continue;
        for (int w = 0; w < W; ++w) {
          H.expn_nib[((size_t)i * 16 + v) * W + w] |= H.exp_n[(size_t)B * W + w];
          H.pred_nib[((size_t)i * 16 + v) * W + w] |= H.pred[(size_t)B * W + w];
        }
      }
  H.lhs_nib.assign((size_t)W * 8 * 16, 0);
  H.sym_nib.assign((size_t)W * 8 * 16 * 2, 0);
  for (int w = 0; w < W; ++w)
    for (int j = 0; j < 8; ++j)
      for (int v = 0; v < 16; ++v)
        for (int b = 0; b < 4; ++b) {
          if (!((v >> b) & 1)) continue;
          const int it = w * 32 + 4 * j + b;
          const size_t e = ((size_t)w * 8 + j) * 16 + v;
          if (((H.complete[w] >> (4 * j + b)) & 1) && H.item_lhs[it] >= 0) H.lhs_nib[e] |= 1ull << H.item_lhs[it];
          const int sym = H.next_sym[it];
          if (sym >= 64)
            H.sym_nib[2 * e] |= 1ull << (sym - 64);
          else if (sym >= 0)
            H.sym_nib[2 * e + 1] |= 1ull << sym;
        }
  H.predsym_nib.assign((size_t)16 * 16 * 2, 0);
  for (int e = 0; e < 16 * 16; ++e)
    for (int w = 0; w < W; ++w)
      for (uint32_t bits = H.pred_nib[(size_t)e * W + w]; bits; bits &= bits - 1) {
        const int sym = H.next_sym[w * 32 + __builtin_ctz(bits)];
        if (sym >= 64)
          H.predsym_nib[2 * e] |= 1ull << (sym - 64);
        else if (sym >= 0)
          H.predsym_nib[2 * e + 1] |= 1ull << sym;
      }

  // ---------------------------------------------------------------- cover
  {
    // epsilon edges of the flattened recursive transition network (App. A.2):
    // entry_A -> (p,0) for A's productions, (p,|rhs|) -> exit_A, a nonterminal
    // B at (p,k): (p,k) -> entry_B and exit_B -> (p,k+1) for every occurrence
    const int CW = H.CW, nbits = CW * 32;
    auto ENT = [&](int A) { return W * 32 + A; };
    auto EXT = [&](int A) { return W * 32 + 64 + A; };
    std::vector<std::vector<int>> eps(nbits);
    for (int p = 0; p < P; ++p) {
      int A = lhs[p] - T, len = roff[p + 1] - roff[p];
      eps[ENT(A)].push_back(base[p]);
      eps[base[p] + len].push_back(EXT(A));
      for (int k = 0; k < len; ++k) {
        int X = rhs[roff[p] + k];
        if (X >= T) {
          eps[base[p] + k].push_back(ENT(X - T));
          eps[EXT(X - T)].push_back(base[p] + k + 1);
        }
      }
    }
    H.cover_cl.assign((size_t)nbits * CW, 0);
    for (int s = 0; s < nbits; ++s) {
      std::vector<char> seen(nbits, 0);
      std::vector<int> st{s};
      seen[s] = 1;
      while (!st.empty()) {
        int u = st.back();
        st.pop_back();
        set32(H.cover_cl, (size_t)s * CW, u);
        for (int v : eps[u])
          if (!seen[v]) {
            seen[v] = 1;
            st.push_back(v);
          }
      }
    }
  }

  // ---------------------------------------------------------------- lexer
  const int QW = H.QW;
  H.ext.assign((size_t)Q * QW, 0);
  for (int q = 0; q < Q; ++q) {
    std::vector<char> seen(Q, 0);
    std::vector<int> st{q};
    seen[q] = 1;
    while (!st.empty()) {
      int u = st.back();
      st.pop_back();
      set32(H.ext, (size_t)q * QW, u);
      for (int c = 0; c < 256; ++c) {
        int d = trans[u * 256 + c];
        if (d >= 0 && !seen[d]) {
          seen[d] = 1;
          st.push_back(d);
        }
      }
    }
  }
  H.flushlab.assign(Q, 0);
  for (int q = 0; q < Q; ++q) {
    if (q == 0 || accept[q] == -2)
      H.flushlab[q] = 1ull << kLabelEps;
    else if (accept[q] >= 0)
      H.flushlab[q] = 1ull << accept[q];
  }
  // fresh states and emissions
  std::vector<int> fresh_id(Q, -1), fresh;
  for (int c = 0; c < 256; ++c) {
    int f = trans[c];
    if (f >= 0 && fresh_id[f] < 0) {
      fresh_id[f] = (int)fresh.size();
      fresh.push_back(f);
    }
  }
  const int F = (int)fresh.size();
  // emit[q][r] = labels emitted when a lexeme ending in state q is followed by
  // a byte that starts fresh state r
  std::vector<std::vector<uint64_t>> emit(Q, std::vector<uint64_t>(F, 0));
  for (int q = 0; q < Q; ++q) {
    if (accept[q] == -1) continue;
    uint64_t lab = accept[q] == -2 ? (1ull << kLabelEps) : (1ull << accept[q]);
    for (int c = 0; c < 256; ++c)
      if (trans[q * 256 + c] < 0 && trans[c] >= 0) emit[q][fresh_id[trans[c]]] |= lab;
  }
  auto in_ext = [&](int q, int u) { return (H.ext[(size_t)q * QW + (u >> 5)] >> (u & 31)) & 1; };
  std::vector<std::vector<uint64_t>> internal(F, std::vector<uint64_t>(F, 0));
  for (int r = 0; r < F; ++r)
    for (int q = 0; q < Q; ++q)
      if (in_ext(fresh[r], q))
        for (int r2 = 0; r2 < F; ++r2) internal[r][r2] |= emit[q][r2];
  std::vector<std::vector<uint64_t>> entry(Q, std::vector<uint64_t>(F, 0));
  for (int qi = 0; qi < Q; ++qi)
    for (int q = 0; q < Q; ++q)
      if (in_ext(qi, q))
        for (int r2 = 0; r2 < F; ++r2) entry[qi][r2] |= emit[q][r2];
  // left-language classes: determinise from every entry state, record subsets
  auto closure = [&](Bits s) {
    bool changed = true;
    while (changed) {
      changed = false;
      for (int r = 0; r < F; ++r)
        if (s.get(r))
          for (int r2 = 0; r2 < F; ++r2)
            if (!s.get(r2) && ((internal[r][r2] >> kLabelEps) & 1)) {
              s.set(r2);
              changed = true;
            }
    }
    return s;
  };
  std::map<Bits, int> subsets;
  for (int qi = 0; qi < Q; ++qi) {
    Bits s0(F);
    for (int r = 0; r < F; ++r)
      if ((entry[qi][r] >> kLabelEps) & 1) s0.set(r);
    s0 = closure(s0);
    std::set<Bits> seen;
    std::vector<std::pair<bool, Bits>> work{{true, s0}};
    if (s0.any()) subsets.emplace(s0, (int)subsets.size());
    std::set<std::pair<bool, Bits>> visited{{true, s0}};
    for (size_t i = 0; i < work.size(); ++i) {
      bool from_entry = work[i].first;
      Bits cur = work[i].second;
      for (int a = 0; a < T; ++a) {
        Bits nx(F);
        for (int r2 = 0; r2 < F; ++r2) {
          bool hit = from_entry && ((entry[qi][r2] >> a) & 1);
          for (int r = 0; r < F && !hit; ++r)
            if (cur.get(r) && ((internal[r][r2] >> a) & 1)) hit = true;
          if (hit) nx.set(r2);
        }
        if (!nx.any()) continue;
        nx = closure(nx);
        if (visited.insert({false, nx}).second) {
          work.push_back({false, nx});
          if (!subsets.count(nx)) subsets.emplace(nx, (int)subsets.size());
        }
      }
    }
  }
  std::map<std::vector<int>, int> sig2class;
  std::vector<int> cls_of(F, -1);
  for (int r = 0; r < F; ++r) {
    std::vector<int> sig;
    for (auto& kv : subsets)
      if (kv.first.get(r)) sig.push_back(kv.second);
    if (sig.empty()) continue;  // never reached inside a gap
    std::sort(sig.begin(), sig.end());
    auto it = sig2class.find(sig);
    if (it == sig2class.end()) {
      int k = (int)sig2class.size();
      sig2class[sig] = k;
      cls_of[r] = k;
    } else {
      cls_of[r] = it->second;
    }
  }
  const int K = (int)sig2class.size();
  if (K > kMaxGapClasses) {
    why = "lexer gap automaton has too many left-language classes";
    return EPIC_ERR_UNSUPPORTED;
  }
  H.K = K;
  H.cls_exit.assign((size_t)std::max(K, 1) * QW, 0);
  H.cls_internal.assign((size_t)std::max(K * K, 1), 0);
  H.cls_entry.assign((size_t)Q * std::max(K, 1), 0);
  H.cls_flush.assign(std::max(K, 1), 0);
  for (int r = 0; r < F; ++r) {
    int k = cls_of[r];
    if (k < 0) continue;
    for (int w = 0; w < QW; ++w) H.cls_exit[(size_t)k * QW + w] |= H.ext[(size_t)fresh[r] * QW + w];
    for (int r2 = 0; r2 < F; ++r2)
      if (cls_of[r2] >= 0) H.cls_internal[(size_t)k * K + cls_of[r2]] |= internal[r][r2];
    for (int qi = 0; qi < Q; ++qi) H.cls_entry[(size_t)qi * K + k] |= entry[qi][r];
  }
  for (int k = 0; k < K; ++k)
    for (int q = 0; q < Q; ++q)
      if ((H.cls_exit[(size_t)k * QW + (q >> 5)] >> (q & 31)) & 1) H.cls_flush[k] |= H.flushlab[q];

  // ---------------------------------------------------------------- gap derivations
  // Inside a masked run the class nodes and their edges do not depend on the
  // sequence, so what the run can derive does not either.  eps_path[j*K+k]:
  // class k is reachable from class j by epsilon edges (reflexive).
  // gap_nt[j*K+k]: nonterminals B with a string of L(B) labelling a path from
  // class j to class k (least fixpoint over the productions, the Bar-Hillel
  // construction restricted to the run's class automaton).
  const int KK = std::max(K, 1);
  std::vector<char> epsp((size_t)KK * KK, 0);
  for (int j = 0; j < K; ++j) epsp[(size_t)j * K + j] = 1;
  for (bool changed = true; changed;) {
    changed = false;
    for (int i = 0; i < K; ++i)
      for (int j = 0; j < K; ++j)
        if (epsp[(size_t)i * K + j])
          for (int k = 0; k < K; ++k)
            if (((H.cls_internal[(size_t)j * K + k] >> kLabelEps) & 1) && !epsp[(size_t)i * K + k]) {
              epsp[(size_t)i * K + k] = 1;
              changed = true;
            }
  }
  std::vector<uint64_t> gnt((size_t)KK * KK, 0);
  for (bool changed = true; changed;) {
    changed = false;
    for (int p = 0; p < P; ++p) {
      const int A = lhs[p] - T;
      for (int j = 0; j < K; ++j) {
        std::vector<char> S(K, 0);
        for (int k = 0; k < K; ++k) S[k] = epsp[(size_t)j * K + k];
        for (int i = roff[p]; i < roff[p + 1]; ++i) {
          const int X = rhs[i];
          std::vector<char> S2(K, 0);
          for (int c = 0; c < K; ++c) {
            if (!S[c]) continue;
            for (int c2 = 0; c2 < K; ++c2) {
              if (X < T) {
                if ((H.cls_internal[(size_t)c * K + c2] >> X) & 1)
                  for (int c3 = 0; c3 < K; ++c3)
                    if (epsp[(size_t)c2 * K + c3]) S2[c3] = 1;
              } else if ((gnt[(size_t)c * K + c2] >> (X - T)) & 1) {
                S2[c2] = 1;
              }
            }
          }
          S = S2;
        }
        for (int k = 0; k < K; ++k)
          if (S[k] && !((gnt[(size_t)j * K + k] >> A) & 1)) {
            gnt[(size_t)j * K + k] |= 1ull << A;
            changed = true;
          }
      }
    }
  }
  // transfer masks between the class nodes of a run: items whose next symbol
  // is a label of an edge j -> k or a nonterminal derivable from j to k
  H.gap_eps = 0;
  H.gap_tm.assign((size_t)KK * KK * W, 0);
  for (int j = 0; j < K; ++j)
    for (int k = 0; k < K; ++k) {
      if (epsp[(size_t)j * K + k]) H.gap_eps |= 1ull << (j * K + k);
      Set m = exp_mask(gnt[(size_t)j * K + k]);
      uint64_t lab = H.cls_internal[(size_t)j * K + k] & ~(1ull << kLabelEps);
      for (int a = 0; a < T; ++a)
        if ((lab >> a) & 1)
          for (int w = 0; w < W; ++w) m[w] |= H.exp_t[(size_t)a * W + w];
      for (int w = 0; w < W; ++w) H.gap_tm[((size_t)j * K + k) * W + w] = m[w];
    }
  H.gap_nt = gnt;
  // Entries of a run's own origins: every production predicted at class node
  // j (predicting everything is sound: an Earley item only asserts that its
  // prefix derives the input it spans), closed under the run's transfers;
  // gap_own[(j*K + k)*W ..] is the item set of the entry of origin j at class k.
  // cover reachability inside a run, by search over (class, cover state)
  {
    const int CW = H.CW, S = CW * 32;
    std::vector<std::vector<int>> ceps(S);
    for (int s = 0; s < S; ++s)
      for (int u = 0; u < S; ++u)
        if (u != s && ((H.cover_cl[(size_t)s * CW + (u >> 5)] >> (u & 31)) & 1)) ceps[s].push_back(u);
    H.gap_cover.assign((size_t)KK * KK * S * CW, 0);
    std::vector<char> seen((size_t)KK * S);
    std::vector<int> stack;
    for (int j = 0; j < K; ++j)
      for (int s0 = 0; s0 < S; ++s0) {
        std::fill(seen.begin(), seen.end(), 0);
        stack.assign(1, j * S + s0);
        seen[(size_t)j * S + s0] = 1;
        while (!stack.empty()) {
          const int node = stack.back();
          stack.pop_back();
          const int c = node / S, st = node % S;
          H.gap_cover[(((size_t)j * K + c) * S + s0) * CW + (st >> 5)] |= 1u << (st & 31);
          auto push = [&](int c2, int s2) {
            if (!seen[(size_t)c2 * S + s2]) {
              seen[(size_t)c2 * S + s2] = 1;
              stack.push_back(c2 * S + s2);
            }
          };
          for (int u : ceps[st]) push(c, u);
          for (int c2 = 0; c2 < K; ++c2) {
            const uint64_t lab = H.cls_internal[(size_t)c * K + c2];
            if ((lab >> kLabelEps) & 1) push(c2, st);
            if (st < ni && H.next_sym[st] >= 0 && H.next_sym[st] < 64 && ((lab >> H.next_sym[st]) & 1)) push(c2, st + 1);
          }
        }
      }
  }
  H.gap_own.assign((size_t)KK * KK * W, 0);
  for (int j = 0; j < K; ++j) {
    std::vector<Set> x(K, Set(W, 0));
    for (int A = 0; A < N; ++A)
      for (int w = 0; w < W; ++w) x[j][w] |= H.start_of[(size_t)A * W + w];
    for (bool changed = true; changed;) {
      changed = false;
      for (int a = 0; a < K; ++a)
        for (int b = 0; b < K; ++b) {
          Set m(H.gap_tm.begin() + ((size_t)a * K + b) * W, H.gap_tm.begin() + ((size_t)a * K + b + 1) * W);
          if (adv_or(x[a], m, x[b])) changed = true;
          if (a != b && epsp[(size_t)a * K + b])
            for (int w = 0; w < W; ++w)
              if (x[a][w] & ~x[b][w]) {
                x[b][w] |= x[a][w];
                changed = true;
              }
        }
    }
    for (int k = 0; k < K; ++k)
      for (int w = 0; w < W; ++w) H.gap_own[((size_t)j * K + k) * W + w] = x[k][w];
  }
  // ---------------------------------------------------------------- witness strings
  H.dot0.assign(W, 0);
  for (int p = 0; p <= P; ++p) set32(H.dot0, 0, base[p]);
  build_witness_strings(H, K, epsp, T, N, P, lhs, roff, rhs, base);
  return 0;
}

}  // namespace epic
