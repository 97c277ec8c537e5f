// EPIC oracle: plain, slow, obviously-correct CPU implementation of the
// validity check and the relaxed compatible-subset selection.
//
// TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
// baseline leg of the benchmark may load this library.  It shares no code,
// header, table or helper with the HIP path; both consume the same lexer DFA,
// grammar and vocabulary arrays produced by the seeded input generators.
//
// What it computes (paper references are to arxiv 2606.00722):
//
//  * greedy lexing step (lexing semantics, reading of Sec. 3 "lexical map"):
//      step(q,c) = (delta(q,c), eps)                  if delta(q,c) defined
//                = (delta(q0,c), [acc(q)] or eps)     if acc(q) set, delta(q0,c) defined
//                                                      (eps when acc(q) is skip)
//                = DEAD                               otherwise
//      flush(q)  = eps (q = q0), [acc(q)] (terminal), eps (skip), DEAD (else)
//  * memo[t][q]: the fold of step over the bytes of token t from state q
//    (Alg. 2's cached span lexing, keyed by token and boundary state).
//  * R_x: the fixed bytes of x with every maximal run of masks replaced by
//    Sigma* over all 256 bytes (Limitations: masks over-approximated by Sigma*).
//  * A_x (Sec. 3, C_x = L(A_x)): the product of R_x's character automaton with
//    the greedy lexer, built directly from the bytes (never from the memo).
//  * Valid(x) = [L(G) cap L(A_x) != empty] (Sec. 3, the completable criterion).
//    Decided by: epsilon-closure subset construction of A_x into a DFA over
//    grammar terminals, Moore minimisation (both language-preserving textbook
//    steps), then a deductive Earley recogniser over the DFA's states (Alg. 3:
//    predict / scan / complete generalised from string positions to graph
//    nodes, applied to a fixpoint; completion in both orders so that nullable
//    nonterminals are handled).
//  * Relaxed(x) = [L(F_G) cap L(A_x) != empty] where F_G is the RTN flattening
//    of G (App. A.2, App. D.3 "Regular Cover"): entry/exit states per
//    nonterminal, one state per rule position, every call site flattened.
//    Decided by breadth-first search of the product with the same DFA.
//  * Witness (Sec. 4, failure recovery: a valid x has a completion, and the
//    output is completed from it): the Bar-Hillel triples of the same DFA
//    (App. A.2), found in rounds so that the expansion of (S, start, final)
//    terminates, give a terminal string of L(G) accepted by A_x; a breadth-first
//    search of A_x finds a path spelling it; its moves inside masked runs give
//    the bytes of each run.
//  * The prior pipeline ("Con.", Sec. 2, App. A.1-A.2), a CPU comparator: the
//    same automaton, determinised, minimised by Hopcroft's algorithm, then the
//    emptiness of its intersection with the grammar (Bar-Hillel facts over a
//    binarised grammar, by an agenda); timed per phase.
//  * Select: Alg. 4 (RelaxedSelect then ExactShrink) over the candidates of a
//    sequence whose individual verdict is 1, sorted by descending float32
//    confidence with ties to the lower candidate index, halves split with the
//    first ceil(|C|/2) candidates on the high-confidence side.
#include <algorithm>
#include <array>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <atomic>
#include <cstdint>
#include <cstring>
#include <deque>
#include <functional>
#include <map>
#include <set>
#include <thread>
#include <unordered_map>
#include <unordered_set>
#include <vector>

namespace {

struct Lexer {
  int Q;
  const int16_t* trans;   // [Q*256], -1 = none
  const int16_t* accept;  // [Q], -1 none, -2 skip, >=0 terminal
};

struct Grammar {
  int T, N, start, P;
  const int32_t* lhs;   // [P]
  const int32_t* roff;  // [P+1]
  const int32_t* rhs;   // symbols: <T terminal, >=T nonterminal
};

struct Vocab {
  int V;
  const uint8_t* bytes;
  const int32_t* offs;  // [V+1]
};

constexpr int kSkip = -2;
constexpr int kNone = -1;
constexpr int kDead = -1;

// ----- greedy lexing step -------------------------------------------------------
// returns next state or kDead; *out = kNone (no emission), kSkip, or terminal id
int lex_step(const Lexer& L, int q, int c, int* out) {
  int d = L.trans[q * 256 + c];
  if (d >= 0) {
    *out = kNone;
    return d;
  }
  int a = L.accept[q];
  int f = L.trans[0 * 256 + c];
  if (a != kNone && f >= 0) {
    *out = a;  // terminal id or kSkip
    return f;
  }
  return kDead;
}

// returns false if DEAD; *out = kNone or terminal
bool lex_flush(const Lexer& L, int q, int* out) {
  if (q == 0) { *out = kNone; return true; }
  int a = L.accept[q];
  if (a >= 0) { *out = a; return true; }
  if (a == kSkip) { *out = kNone; return true; }
  return false;
}

// ----- character-level product automaton A_x -----------------------------------
// A slot is a fixed byte (0..255) or a gap (-1).  Node (s, q) = id s*Q + q for
// slots s in [0, S]; slot S is the end.  FINAL = (S+1)*Q.
struct CharNFA {
  int Q = 0, S = 0, final_node = 0;
  std::vector<int> slot;  // [S]
  // adjacency, only for nodes that are reachable from the start
  std::vector<std::vector<int>> eps;                         // eps successors
  std::vector<std::vector<std::pair<int, int>>> lab;         // (terminal, successor)
  std::vector<char> alive;                                   // reachable & co-reachable
};

std::vector<int> make_slots(const Vocab& V, const int32_t* x, int n) {
  std::vector<int> slots;
  for (int i = 0; i < n; ++i) {
    if (x[i] < 0) {
      if (slots.empty() || slots.back() != -1) slots.push_back(-1);
    } else {
      for (int j = V.offs[x[i]]; j < V.offs[x[i] + 1]; ++j) slots.push_back(V.bytes[j]);
    }
  }
  return slots;
}

void build_char_nfa(const Lexer& L, const std::vector<int>& slots, CharNFA& A) {
  A.Q = L.Q;
  A.S = (int)slots.size();
  A.slot = slots;
  int nnodes = (A.S + 1) * A.Q + 1;
  A.final_node = nnodes - 1;
  A.eps.assign(nnodes, {});
  A.lab.assign(nnodes, {});
  std::vector<char> seen(nnodes, 0);
  std::vector<int> stack;
  auto push = [&](int v) {
    if (!seen[v]) { seen[v] = 1; stack.push_back(v); }
  };
  auto add = [&](int u, int o, int v) {
    if (o == kNone || o == kSkip) A.eps[u].push_back(v);
    else A.lab[u].push_back({o, v});
    push(v);
  };
  push(0 * A.Q + 0);
  while (!stack.empty()) {
    int u = stack.back();
    stack.pop_back();
    if (u == A.final_node) continue;
    int s = u / A.Q, q = u % A.Q;
    if (s == A.S) {
      int o;
      if (lex_flush(L, q, &o)) add(u, o, A.final_node);
      continue;
    }
    int c = A.slot[s];
    if (c >= 0) {
      int o;
      int q2 = lex_step(L, q, c, &o);
      if (q2 != kDead) add(u, o, (s + 1) * A.Q + q2);
    } else {
      add(u, kNone, (s + 1) * A.Q + q);  // leave the gap
      for (int b = 0; b < 256; ++b) {    // one more byte inside the gap
        int o;
        int q2 = lex_step(L, q, b, &o);
        if (q2 != kDead) add(u, o, s * A.Q + q2);
      }
    }
  }
  // many bytes lead to the same successor inside a gap: keep each edge once
  for (int u = 0; u < nnodes; ++u) {
    if (!seen[u]) continue;
    std::sort(A.eps[u].begin(), A.eps[u].end());
    A.eps[u].erase(std::unique(A.eps[u].begin(), A.eps[u].end()), A.eps[u].end());
    std::sort(A.lab[u].begin(), A.lab[u].end());
    A.lab[u].erase(std::unique(A.lab[u].begin(), A.lab[u].end()), A.lab[u].end());
  }
  // co-reachability (reverse search from FINAL)
  std::vector<std::vector<int>> rev(nnodes);
  for (int u = 0; u < nnodes; ++u) {
    if (!seen[u]) continue;
    for (int v : A.eps[u]) rev[v].push_back(u);
    for (auto& e : A.lab[u]) rev[e.second].push_back(u);
  }
  A.alive.assign(nnodes, 0);
  if (seen[A.final_node]) {
    std::vector<int> st{A.final_node};
    A.alive[A.final_node] = 1;
    while (!st.empty()) {
      int v = st.back();
      st.pop_back();
      for (int u : rev[v])
        if (!A.alive[u]) { A.alive[u] = 1; st.push_back(u); }
    }
  }
}

// ----- DFA over grammar terminals -------------------------------------------
struct DFA {
  int T = 0;
  int start = -1;                 // -1: empty language
  std::vector<std::vector<int>> trans;  // [state][T], -1 = none
  std::vector<char> fin;
  int states() const { return (int)trans.size(); }
};

// in-place epsilon closure of a duplicate-free node set; `mark` is a scratch
// array of A's size that is all zero on entry and on return
void eps_closure(const CharNFA& A, std::vector<int>& set, std::vector<char>& mark) {
  for (int u : set) mark[u] = 1;
  for (size_t i = 0; i < set.size(); ++i)
    for (int v : A.eps[set[i]])
      if (A.alive[v] && !mark[v]) { mark[v] = 1; set.push_back(v); }
  for (int u : set) mark[u] = 0;
  std::sort(set.begin(), set.end());
}

struct VecHash {
  size_t operator()(const std::vector<int>& v) const {
    uint64_t h = 1469598103934665603ull;
    for (int x : v) h = (h ^ (uint64_t)x) * 1099511628211ull;
    return (size_t)h;
  }
};

// Epsilon removal followed by subset construction.  The states of the
// epsilon-free automaton are the start node and every target of a labelled
// edge; node u gets an edge (a, v) whenever v follows a labelled edge a from
// some node of u's epsilon closure, and accepts when FINAL is in that closure.
// Subsets of these states are then determinised over the grammar terminals.
// Returns false if the DFA state limit is exceeded.
bool determinize(const CharNFA& A, int T, DFA& D, size_t limit) {
  D = DFA();
  D.T = T;
  if (!A.alive[0]) return true;  // empty language
  const int nn = (int)A.alive.size();
  std::vector<char> is_item(nn, 0);
  is_item[0] = 1;
  for (int u = 0; u < nn; ++u)
    if (A.alive[u])
      for (auto& e : A.lab[u])
        if (A.alive[e.second]) is_item[e.second] = 1;
  std::vector<char> mark(nn, 0);
  std::vector<std::vector<std::pair<int, int>>> out(nn);  // (terminal, item node), epsilon-free
  std::vector<char> fin(nn, 0);
  for (int u = 0; u < nn; ++u) {
    if (!is_item[u]) continue;
    std::vector<int> cl{u};
    eps_closure(A, cl, mark);
    for (int w : cl) {
      if (w == A.final_node) fin[u] = 1;
      for (auto& e : A.lab[w])
        if (A.alive[e.second]) out[u].push_back(e);
    }
    std::sort(out[u].begin(), out[u].end());
    out[u].erase(std::unique(out[u].begin(), out[u].end()), out[u].end());
  }
  std::unordered_map<std::vector<int>, int, VecHash> ids;
  std::vector<std::vector<int>> order;
  ids[{0}] = 0;
  order.push_back({0});
  for (size_t i = 0; i < order.size(); ++i) {
    if (order.size() > limit) return false;
    std::vector<std::vector<int>> moves(T);
    for (int u : order[i])
      for (auto& e : out[u]) moves[e.first].push_back(e.second);
    std::vector<int> row(T, -1);
    for (int a = 0; a < T; ++a) {
      if (moves[a].empty()) continue;
      std::sort(moves[a].begin(), moves[a].end());
      moves[a].erase(std::unique(moves[a].begin(), moves[a].end()), moves[a].end());
      auto it = ids.find(moves[a]);
      int id;
      if (it == ids.end()) {
        id = (int)order.size();
        ids[moves[a]] = id;
        order.push_back(moves[a]);
      } else {
        id = it->second;
      }
      row[a] = id;
    }
    D.trans.push_back(row);
  }
  D.fin.assign(order.size(), 0);
  for (size_t i = 0; i < order.size(); ++i)
    for (int u : order[i]) D.fin[i] |= fin[u];
  D.start = 0;
  return true;
}

// Moore partition refinement (missing transitions go to an implicit dead block)
void minimize(DFA& D) {
  int n = D.states();
  if (n == 0) return;
  std::vector<int> block(n);
  for (int i = 0; i < n; ++i) block[i] = D.fin[i] ? 1 : 0;
  int nb = 0;
  while (true) {
    std::map<std::vector<int>, int> sig;
    std::vector<int> nbk(n);
    for (int i = 0; i < n; ++i) {
      std::vector<int> s;
      s.reserve(D.T + 1);
      s.push_back(block[i]);
      for (int a = 0; a < D.T; ++a) s.push_back(D.trans[i][a] < 0 ? -1 : block[D.trans[i][a]]);
      auto it = sig.find(s);
      if (it == sig.end()) {
        int id = (int)sig.size();
        sig[s] = id;
        nbk[i] = id;
      } else {
        nbk[i] = it->second;
      }
    }
    int cnt = (int)sig.size();
    block = nbk;
    if (cnt == nb) break;
    nb = cnt;
  }
  DFA M;
  M.T = D.T;
  M.trans.assign(nb, std::vector<int>(D.T, -1));
  M.fin.assign(nb, 0);
  for (int i = 0; i < n; ++i) {
    int b = block[i];
    M.fin[b] = D.fin[i];
    for (int a = 0; a < D.T; ++a) M.trans[b][a] = D.trans[i][a] < 0 ? -1 : block[D.trans[i][a]];
  }
  M.start = block[D.start];
  D = M;
}

// A_x as a minimal DFA; returns false on blow-up
bool completion_dfa(const Lexer& L, const Grammar& G, const Vocab& V, const int32_t* x, int n, DFA& D) {
  CharNFA A;
  build_char_nfa(L, make_slots(V, x, n), A);
  if (!determinize(A, G.T, D, 4000000)) return false;
  if (D.start >= 0) minimize(D);
  return true;
}

// ----- Earley recogniser over a DFA (Alg. 3, deductive fixpoint) --------------------
struct GrammarView {
  // productions 0..P-1 as given; production P is S' -> S
  int T, N, P;
  std::vector<int> lhs;
  std::vector<std::vector<int>> rhs;
  std::vector<std::vector<int>> by_lhs;  // nonterminal index (0..N-1) -> productions
  explicit GrammarView(const Grammar& G) : T(G.T), N(G.N), P(G.P) {
    lhs.resize(P + 1);
    rhs.resize(P + 1);
    by_lhs.assign(N, {});
    for (int p = 0; p < P; ++p) {
      lhs[p] = G.lhs[p];
      rhs[p].assign(G.rhs + G.roff[p], G.rhs + G.roff[p + 1]);
      by_lhs[G.lhs[p] - G.T].push_back(p);
    }
    lhs[P] = -1;
    rhs[P] = {G.start};
  }
};

bool earley_accepts(const GrammarView& g, const DFA& D) {
  if (D.start < 0) return false;
  // item = (prod, dot, origin, node) packed into 64 bits
  // 16 bits production, 8 bits dot, 20 bits origin, 20 bits node
  auto pack = [](uint64_t p, uint64_t k, uint64_t o, uint64_t v) {
    return (p << 48) | (k << 40) | (o << 20) | v;
  };
  if (D.states() >= (1 << 20) || g.P >= (1 << 16)) return false;
  std::unordered_set<uint64_t> visited;
  std::vector<uint64_t> work;
  // waiting[(node, B)] = items (p,k,o) at node whose next symbol is B
  std::unordered_map<uint64_t, std::vector<uint64_t>> waiting;
  // completed[(origin, B)] = end nodes v of a derivation of B from origin
  std::unordered_map<uint64_t, std::vector<int>> completed;
  std::unordered_set<uint64_t> completed_seen;
  auto key = [](uint64_t node, uint64_t B) { return (node << 20) | B; };
  auto add = [&](int p, int k, int o, int v) {
    uint64_t it = pack(p, k, o, v);
    if (visited.insert(it).second) work.push_back(it);
  };
  const int s = D.start;
  add(g.P, 0, s, s);
  while (!work.empty()) {
    uint64_t it = work.back();
    work.pop_back();
    int p = (int)(it >> 48), k = (int)((it >> 40) & 0xFF), o = (int)((it >> 20) & 0xFFFFF),
        v = (int)(it & 0xFFFFF);
    if (p == g.P && k == 1 && o == s && D.fin[v]) return true;  // S' -> S . from start to a final node
    const auto& r = g.rhs[p];
    if (k < (int)r.size()) {
      int X = r[k];
      if (X < g.T) {  // scan along DFA edges labelled X
        int v2 = D.trans[v][X];
        if (v2 >= 0) add(p, k + 1, o, v2);
      } else {
        int B = X - g.T;
        waiting[key(v, B)].push_back(pack(p, k, o, 0));
        for (int q : g.by_lhs[B]) add(q, 0, v, v);  // predict
        auto c = completed.find(key(v, B));         // complete (completed item seen first)
        if (c != completed.end())
          for (int v2 : c->second) add(p, k + 1, o, v2);
      }
    } else if (p != g.P) {
      int B = g.lhs[p] - g.T;
      uint64_t ck = key(o, B);
      if (completed_seen.insert((ck << 20) | (uint64_t)v).second) {
        completed[ck].push_back(v);
        auto w = waiting.find(ck);  // complete (waiting item seen first)
        if (w != waiting.end())
          for (uint64_t wi : w->second)
            add((int)(wi >> 48), (int)((wi >> 40) & 0xFF) + 1, (int)((wi >> 20) & 0xFFFFF), v);
      }
    }
  }
  return false;
}

// ----- regular cover F_G and the relaxed check -----------------------------------
struct Cover {
  // states: in_A = A, out_A = N + A (A in 0..N-1), rule position (p,k) = 2N + base[p] + k
  int N = 0, nstates = 0, start = 0, accept = 0;
  std::vector<std::vector<int>> eps;
  std::vector<std::vector<std::pair<int, int>>> lab;  // (terminal, successor)
};

Cover build_cover(const Grammar& G) {
  Cover F;
  F.N = G.N;
  std::vector<int> base(G.P + 1);
  int tot = 0;
  for (int p = 0; p < G.P; ++p) {
    base[p] = tot;
    tot += G.roff[p + 1] - G.roff[p] + 1;
  }
  F.nstates = 2 * G.N + tot;
  F.eps.assign(F.nstates, {});
  F.lab.assign(F.nstates, {});
  auto in_ = [&](int A) { return A; };
  auto out_ = [&](int A) { return G.N + A; };
  auto pos = [&](int p, int k) { return 2 * G.N + base[p] + k; };
  for (int p = 0; p < G.P; ++p) {
    int A = G.lhs[p] - G.T;
    int len = G.roff[p + 1] - G.roff[p];
    F.eps[in_(A)].push_back(pos(p, 0));
    F.eps[pos(p, len)].push_back(out_(A));
    for (int k = 0; k < len; ++k) {
      int X = G.rhs[G.roff[p] + k];
      if (X < G.T) {
        F.lab[pos(p, k)].push_back({X, pos(p, k + 1)});
      } else {
        int B = X - G.T;
        F.eps[pos(p, k)].push_back(in_(B));      // call: forget the call site
        F.eps[out_(B)].push_back(pos(p, k + 1));  // return to every continuation
      }
    }
  }
  F.start = in_(G.start - G.T);
  F.accept = out_(G.start - G.T);
  return F;
}

bool cover_accepts(const Cover& F, const DFA& D) {
  if (D.start < 0) return false;
  int nd = D.states();
  std::vector<char> seen((size_t)F.nstates * nd, 0);
  std::deque<std::pair<int, int>> q;
  auto push = [&](int c, int d) {
    size_t k = (size_t)c * nd + d;
    if (!seen[k]) { seen[k] = 1; q.push_back({c, d}); }
  };
  push(F.start, D.start);
  while (!q.empty()) {
    auto [c, d] = q.front();
    q.pop_front();
    if (c == F.accept && D.fin[d]) return true;
    for (int c2 : F.eps[c]) push(c2, d);
    for (auto& e : F.lab[c]) {
      int d2 = D.trans[d][e.first];
      if (d2 >= 0) push(e.second, d2);
    }
  }
  return false;
}

// ----- the prior pipeline ("Con."), a CPU comparator ---------------------------------
// The earlier CFG-constrained decoder (Sec. 2; App. A.1-A.2) re-checks every
// update from scratch: the lexing automaton of the partial output (an
// epsilon-NFA over terminals, built here as for A_x), its determinisation
// (subset construction) and minimisation (Hopcroft's partition refinement,
// O(|Sigma| |Q| log |Q|)), then the emptiness of the intersection of the DFA
// with the grammar (Bar-Hillel: facts (A, p, q), cubic in the DFA states).
// The three phases are timed separately (the Lex / DFA / Val columns of
// Tab. 2).  The verdict is the same criterion as Valid.

// Hopcroft minimisation of D (missing transitions go to an implicit dead state)
void hopcroft_minimize(DFA& D) {
  const int n = D.states(), T = D.T, dead = n, m = n + 1;
  if (n == 0) return;
  auto tr = [&](int s, int a) { return s == dead ? dead : (D.trans[s][a] < 0 ? dead : D.trans[s][a]); };
  // predecessors per (state, terminal)
  std::vector<std::vector<std::vector<int>>> pre(T, std::vector<std::vector<int>>(m));
  for (int st = 0; st < m; ++st)
    for (int a = 0; a < T; ++a) pre[a][tr(st, a)].push_back(st);
  std::vector<int> block(m);
  std::vector<std::vector<int>> blocks;
  std::vector<int> acc, rej;
  for (int st = 0; st < m; ++st) (st < n && D.fin[st] ? acc : rej).push_back(st);
  for (auto* part : {&acc, &rej})
    if (!part->empty()) {
      for (int st : *part) block[st] = (int)blocks.size();
      blocks.push_back(*part);
    }
  std::deque<std::pair<int, int>> work;  // (block, terminal) splitters
  std::set<std::pair<int, int>> in_work;
  const int first = blocks.size() == 2 && blocks[0].size() > blocks[1].size() ? 1 : 0;
  for (int a = 0; a < T; ++a) {
    work.push_back({first, a});
    in_work.insert({first, a});
  }
  while (!work.empty()) {
    const auto [sb, a] = work.front();
    work.pop_front();
    in_work.erase({sb, a});
    // X = states with an a-move into block sb
    std::map<int, std::vector<int>> hit;  // block -> its states in X
    for (int st : blocks[sb])
      for (int pst : pre[a][st]) hit[block[pst]].push_back(pst);
    for (auto& kv : hit) {
      const int y = kv.first;
      std::vector<int>& inx = kv.second;
      std::sort(inx.begin(), inx.end());
      inx.erase(std::unique(inx.begin(), inx.end()), inx.end());
      if (inx.size() == blocks[y].size()) continue;  // no split
      std::set<int> xs(inx.begin(), inx.end());
      std::vector<int> rest;
      for (int st : blocks[y])
        if (!xs.count(st)) rest.push_back(st);
      const int z = (int)blocks.size();
      blocks[y] = inx;
      blocks.push_back(rest);
      for (int st : rest) block[st] = z;
      for (int b = 0; b < T; ++b) {
        if (in_work.count({y, b})) {
          work.push_back({z, b});
          in_work.insert({z, b});
        } else {
          const int small = blocks[y].size() <= blocks[z].size() ? y : z;
          work.push_back({small, b});
          in_work.insert({small, b});
        }
      }
    }
  }
  // the minimal DFA: blocks reachable from the start, without the dead block
  const int dead_block = block[dead];
  std::vector<int> id(blocks.size(), -1);
  std::vector<int> order{block[D.start]};
  id[block[D.start]] = 0;
  DFA M;
  M.T = T;
  for (size_t k = 0; k < order.size(); ++k) {
    const int bl = order[k], rep = blocks[bl][0];
    std::vector<int> row(T, -1);
    for (int a = 0; a < T; ++a) {
      const int to = block[tr(rep, a)];
      if (to == dead_block) continue;
      if (id[to] < 0) {
        id[to] = (int)order.size();
        order.push_back(to);
      }
      row[a] = id[to];
    }
    M.trans.push_back(row);
    M.fin.push_back(rep < n && D.fin[rep]);
  }
  M.start = block[D.start] == dead_block ? -1 : 0;
  if (M.start < 0) M = DFA{T, -1, {}, {}};
  D = M;
}

// Emptiness of the intersection of L(G) and L(D): facts (X, p, q), symbol X
// deriving a string that takes D from p to q, over the grammar binarised
// (A -> X1 X2 ... Xk as a left-nested chain of fresh symbols), by an agenda.
bool intersection_nonempty(const GrammarView& g, const DFA& D) {
  if (D.start < 0) return false;
  const int n = D.states(), T = g.T;
  int nsym = T + g.N;
  std::vector<std::pair<int, int>> unit;              // (A, X): A -> X
  std::vector<std::array<int, 3>> bin;                 // (A, X, Y): A -> X Y
  std::vector<int> eps_nt;
  for (int pr = 0; pr < g.P; ++pr) {
    const int A = g.lhs[pr];
    const auto& r = g.rhs[pr];
    if (r.empty()) {
      eps_nt.push_back(A);
    } else if (r.size() == 1) {
      unit.push_back({A, r[0]});
    } else {
      int left = r[0];
      for (size_t k = 1; k < r.size(); ++k) {
        const int to = k + 1 == r.size() ? A : nsym++;
        bin.push_back({to, left, r[k]});
        left = to;
      }
    }
  }
  std::vector<std::vector<int>> by_unit(nsym), by_left(nsym), by_right(nsym);
  for (size_t k = 0; k < unit.size(); ++k) by_unit[unit[k].second].push_back((int)k);
  for (size_t k = 0; k < bin.size(); ++k) {
    by_left[bin[k][1]].push_back((int)k);
    by_right[bin[k][2]].push_back((int)k);
  }
  std::unordered_set<uint64_t> seen;
  std::vector<std::vector<std::vector<int>>> out(nsym), in(nsym);  // [X][p] -> q, [X][q] -> p
  std::vector<std::array<int, 3>> agenda;
  auto add = [&](int X, int p, int q) {
    const uint64_t key = ((uint64_t)X * n + p) * n + q;
    if (!seen.insert(key).second) return;
    if (out[X].empty()) {
      out[X].assign(n, {});
      in[X].assign(n, {});
    }
    out[X][p].push_back(q);
    in[X][q].push_back(p);
    agenda.push_back({X, p, q});
  };
  for (int p = 0; p < n; ++p) {
    for (int a = 0; a < T; ++a)
      if (D.trans[p][a] >= 0) add(a, p, D.trans[p][a]);
    for (int A : eps_nt) add(A, p, p);
  }
  const int S = g.rhs[g.P][0];
  while (!agenda.empty()) {
    const auto f = agenda.back();
    agenda.pop_back();
    const int X = f[0], p = f[1], q = f[2];
    if (X == S && p == D.start && D.fin[q]) return true;
    for (int k : by_unit[X]) add(unit[k].first, p, q);
    for (int k : by_left[X]) {  // A -> X Y
      const int Y = bin[k][2];
      if (!out[Y].empty())
        for (size_t t = 0; t < out[Y][q].size(); ++t) add(bin[k][0], p, out[Y][q][t]);
    }
    for (int k : by_right[X]) {  // A -> Y X
      const int Y = bin[k][1];
      if (!in[Y].empty())
        for (size_t t = 0; t < in[Y][p].size(); ++t) add(bin[k][0], in[Y][p][t], q);
    }
  }
  return false;
}

// The prior pipeline on x: 1 / 0, or -3 on the DFA limit; ms[0..2] += the
// lexing-automaton, determinise-and-minimise and intersection times.
int con_check(const Lexer& L, const Grammar& G, const Vocab& V, const std::vector<int32_t>& x, double* ms,
              int* dfa_states = nullptr) {
  using clk = std::chrono::steady_clock;
  const auto t0 = clk::now();
  CharNFA A;
  build_char_nfa(L, make_slots(V, x.data(), (int)x.size()), A);
  const auto t1 = clk::now();
  DFA D;
  if (!determinize(A, G.T, D, 4000000)) return -3;
  if (D.start >= 0) hopcroft_minimize(D);
  const auto t2 = clk::now();
  if (dfa_states) *dfa_states = D.start < 0 ? 0 : D.states();
  GrammarView g(G);
  const bool ok = intersection_nonempty(g, D);
  const auto t3 = clk::now();
  if (ms) {
    ms[0] += std::chrono::duration<double, std::milli>(t1 - t0).count();
    ms[1] += std::chrono::duration<double, std::milli>(t2 - t1).count();
    ms[2] += std::chrono::duration<double, std::milli>(t3 - t2).count();
  }
  return ok ? 1 : 0;
}

// ----- per-sequence checks --------------------------------------------------------
// 1 / 0, or -3 when the DFA construction exceeded its state limit
int valid_seq(const Lexer& L, const Grammar& G, const Vocab& V, const std::vector<int32_t>& x) {
  DFA D;
  if (!completion_dfa(L, G, V, x.data(), (int)x.size(), D) || D.states() >= (1 << 20)) return -3;
  GrammarView g(G);
  return earley_accepts(g, D) ? 1 : 0;
}

int relaxed_seq(const Lexer& L, const Grammar& G, const Vocab& V, const std::vector<int32_t>& x) {
  DFA D;
  if (!completion_dfa(L, G, V, x.data(), (int)x.size(), D)) return -3;
  return cover_accepts(build_cover(G), D) ? 1 : 0;
}

// ----- witness: a completion of x (Sec. 4, failure recovery) ---------------------
// Bar-Hillel triples (B, p, q) of a terminal DFA D: nonterminal B derives a
// terminal string that takes D from state p to state q (the intersection
// construction behind the completable criterion, App. A.2).  Found in rounds:
// a triple found in round r keeps its production and the DFA states between
// its symbols, built from terminal moves and triples of rounds before r only,
// so that expanding a triple into a string terminates.
struct Triples {
  struct Rec {
    int round, prod;
    std::vector<int> states;  // |rhs| + 1 states, first = p, last = q
  };
  int N = 0, D = 0;
  std::unordered_map<uint64_t, Rec> rec;
  std::vector<std::vector<std::pair<int, int>>> out;  // [B * D + p]: (q, round)
  uint64_t key(int B, int p, int q) const { return ((uint64_t)B * D + p) * D + q; }
  const Rec* find(int B, int p, int q) const {
    auto it = rec.find(key(B, p, q));
    return it == rec.end() ? nullptr : &it->second;
  }
};

// returns false when D has more than `limit` states
bool bar_hillel_triples(const GrammarView& g, const DFA& D, Triples& T, int limit) {
  T = Triples();
  T.N = g.N;
  T.D = D.states();
  if (T.D > limit) return false;
  T.out.assign((size_t)g.N * T.D, {});
  for (int round = 1;; ++round) {
    std::vector<std::pair<uint64_t, Triples::Rec>> found;
    for (int pr = 0; pr < g.P; ++pr) {
      const int B = g.lhs[pr] - g.T;
      const auto& r = g.rhs[pr];
      for (int p = 0; p < T.D; ++p) {
        // layer[i]: state after i symbols -> state after i - 1 symbols
        std::vector<std::map<int, int>> layer(r.size() + 1);
        layer[0][p] = -1;
        for (size_t i = 0; i < r.size(); ++i) {
          const int X = r[i];
          for (auto& kv : layer[i]) {
            const int st = kv.first;
            if (X < g.T) {
              const int nx = D.trans[st][X];
              if (nx >= 0 && !layer[i + 1].count(nx)) layer[i + 1][nx] = st;
            } else {
              for (auto& qr : T.out[(size_t)(X - g.T) * T.D + st])
                if (qr.second < round && !layer[i + 1].count(qr.first)) layer[i + 1][qr.first] = st;
            }
          }
          if (layer[i + 1].empty()) break;
        }
        for (auto& kv : layer[r.size()]) {
          const int q = kv.first;
          if (T.rec.count(T.key(B, p, q))) continue;
          Triples::Rec rc{round, pr, std::vector<int>(r.size() + 1)};
          int st = q;
          for (size_t i = r.size(); i > 0; --i) {
            rc.states[i] = st;
            st = layer[i][st];
          }
          rc.states[0] = p;
          found.push_back({T.key(B, p, q), rc});
        }
      }
    }
    int added = 0;
    for (auto& f : found) {
      if (T.rec.count(f.first)) continue;  // the same triple from two productions in one round
      const int B = (int)(f.first / ((uint64_t)T.D * T.D)), p = (int)(f.first / T.D % T.D), q = (int)(f.first % T.D);
      T.out[(size_t)B * T.D + p].push_back({q, round});
      T.rec.emplace(f.first, std::move(f.second));
      ++added;
    }
    if (!added) break;
  }
  return true;
}

// The terminal string of triple (B, p, q), appended to w.
void expand_triple(const GrammarView& g, const Triples& T, int B, int p, int q, std::vector<int>& w) {
  const Triples::Rec* rc = T.find(B, p, q);
  const auto& r = g.rhs[rc->prod];
  for (size_t i = 0; i < r.size(); ++i) {
    if (r[i] < g.T)
      w.push_back(r[i]);
    else
      expand_triple(g, T, r[i] - g.T, rc->states[i], rc->states[i + 1], w);
  }
}

// Witness of x: 1 with the bytes of every maximal masked run (in order) in
// gaps, 0 when x is not valid, -3 when a construction limit is exceeded.
int witness_seq(const Lexer& L, const Grammar& G, const Vocab& V, const std::vector<int32_t>& x,
                std::vector<std::vector<uint8_t>>& gaps) {
  gaps.clear();
  const std::vector<int> slots = make_slots(V, x.data(), (int)x.size());
  CharNFA A;
  build_char_nfa(L, slots, A);
  DFA D;
  if (!determinize(A, G.T, D, 4000000)) return -3;
  if (D.start < 0) return 0;
  minimize(D);
  GrammarView g(G);
  Triples T;
  if (!bar_hillel_triples(g, D, T, 20000)) return -3;
  int fin = -1;
  for (int f = 0; f < D.states() && fin < 0; ++f)
    if (D.fin[f] && T.find(G.start - G.T, D.start, f)) fin = f;
  if (fin < 0) return 0;
  std::vector<int> w;
  expand_triple(g, T, G.start - G.T, D.start, fin, w);
  // a path of A_x spelling w: breadth-first over (node, symbols read)
  const int nn = (int)A.alive.size(), m = (int)w.size();
  auto id = [m](int u, int i) { return (int64_t)u * (m + 1) + i; };
  std::unordered_map<int64_t, int64_t> pred;
  std::deque<int64_t> queue;
  const int64_t s0 = id(0, 0), goal = id(A.final_node, m);
  pred[s0] = -1;
  queue.push_back(s0);
  while (!queue.empty() && !pred.count(goal)) {
    const int64_t cur = queue.front();
    queue.pop_front();
    const int u = (int)(cur / (m + 1)), i = (int)(cur % (m + 1));
    auto visit = [&](int v, int j) {
      if (v < 0 || v >= nn || !A.alive[v]) return;
      const int64_t nx = id(v, j);
      if (pred.emplace(nx, cur).second) queue.push_back(nx);
    };
    for (int v : A.eps[u]) visit(v, i);
    if (i < m)
      for (auto& e : A.lab[u])
        if (e.first == w[i]) visit(e.second, i + 1);
  }
  if (!pred.count(goal)) return -3;  // cannot happen: D and A_x have the same language
  std::vector<int64_t> path;
  for (int64_t c = goal; c >= 0; c = pred[c]) path.push_back(c);
  std::reverse(path.begin(), path.end());
  // bytes of the moves inside masked runs
  std::vector<int> gap_of(slots.size() + 1, -1);
  int ng = 0;
  for (size_t k = 0; k < slots.size(); ++k)
    if (slots[k] == -1) gap_of[k] = ng++;
  gaps.assign(ng, {});
  for (size_t k = 0; k + 1 < path.size(); ++k) {
    const int u = (int)(path[k] / (m + 1)), v = (int)(path[k + 1] / (m + 1));
    const bool labelled = path[k + 1] % (m + 1) != path[k] % (m + 1);
    if (u == A.final_node || v == A.final_node) continue;
    const int su = u / A.Q, qu = u % A.Q, sv = v / A.Q, qv = v % A.Q;
    if (su >= A.S || slots[su] != -1 || sv != su) continue;  // fixed byte, or leaving the run
    int byte = -1;
    for (int c = 0; c < 256 && byte < 0; ++c) {
      int o;
      const int q2 = lex_step(L, qu, c, &o);
      if (q2 != qv) continue;
      const bool emits = o != kNone && o != kSkip;
      if (labelled ? (emits && o == w[path[k] % (m + 1)]) : !emits) byte = c;
    }
    if (byte < 0) return -3;  // cannot happen: the move was made by some byte
    gaps[gap_of[su]].push_back((uint8_t)byte);
  }
  return 1;
}

struct Cand {
  int idx, pos, tok;
  float conf;
};

std::vector<int32_t> apply_cands(const std::vector<int32_t>& x, const std::vector<Cand>& S) {
  std::vector<int32_t> y = x;
  for (const Cand& c : S) y[c.pos] = c.tok;
  return y;
}

struct Selector {
  const Lexer& L;
  const Grammar& G;
  const Vocab& V;
  long cover_calls = 0, exact_calls = 0;
  int err = 0;

  static void halves(const std::vector<Cand>& C, std::vector<Cand>& a, std::vector<Cand>& b) {
    size_t h = (C.size() + 1) / 2;  // ceil(|C|/2) on the high-confidence side
    a.assign(C.begin(), C.begin() + h);
    b.assign(C.begin() + h, C.end());
  }
  static std::vector<Cand> cat(const std::vector<Cand>& a, const std::vector<Cand>& b) {
    std::vector<Cand> r = a;
    r.insert(r.end(), b.begin(), b.end());
    return r;
  }

  std::vector<Cand> relaxed_select(const std::vector<int32_t>& x, const std::vector<Cand>& C) {
    if (C.size() <= 1) return {};
    ++cover_calls;
    int r = relaxed_seq(L, G, V, apply_cands(x, C));
    if (r < 0) { err = r; return {}; }
    if (r) return C;
    std::vector<Cand> CL, CR;
    halves(C, CL, CR);
    std::vector<Cand> BL = relaxed_select(x, CL);
    std::vector<Cand> BR = relaxed_select(apply_cands(x, BL), CR);
    return cat(BL, BR);
  }

  std::vector<Cand> exact_shrink(const std::vector<int32_t>& x, const std::vector<Cand>& B) {
    if (B.size() <= 1) return {};
    ++exact_calls;
    int r = valid_seq(L, G, V, apply_cands(x, B));
    if (r < 0) { err = r; return {}; }
    if (r) return B;
    std::vector<Cand> BL, BR;
    halves(B, BL, BR);
    std::vector<Cand> BL1 = exact_shrink(x, BL);
    std::vector<int32_t> x1 = apply_cands(x, BL1);
    std::vector<Cand> BR1 = relaxed_select(x1, BR);
    std::vector<Cand> BR2 = exact_shrink(x1, BR1);
    return cat(BL1, BR2);
  }
};

void run_parallel(int count, int nthreads, const std::function<void(int)>& fn) {
  if (nthreads <= 1 || count <= 1) {
    for (int i = 0; i < count; ++i) fn(i);
    return;
  }
  std::atomic<int> next{0};
  std::vector<std::thread> ts;
  for (int t = 0; t < nthreads; ++t)
    ts.emplace_back([&]() {
      for (int i; (i = next.fetch_add(1)) < count;) fn(i);
    });
  for (auto& t : ts) t.join();
}
}  // namespace

extern "C" {

typedef struct {
  int32_t num_states;
  const int16_t* trans;
  const int16_t* accept;
} oracle_lexer;
typedef struct {
  int32_t num_terminals, num_nonterminals, start, num_productions;
  const int32_t *lhs, *rhs_offsets, *rhs;
} oracle_grammar;
typedef struct {
  int32_t vocab_size;
  const uint8_t* bytes;
  const int32_t* offsets;
} oracle_vocab;

static Lexer to_lexer(const oracle_lexer* l) { return Lexer{l->num_states, l->trans, l->accept}; }
static Grammar to_grammar(const oracle_grammar* g) {
  return Grammar{g->num_terminals, g->num_nonterminals, g->start, g->num_productions, g->lhs, g->rhs_offsets, g->rhs};
}
static Vocab to_vocab(const oracle_vocab* v) { return Vocab{v->vocab_size, v->bytes, v->offsets}; }

// One greedy step: returns the next state or -1 (dead); *emit = -1 none, -2 skip, >=0 terminal.
int oracle_lex_step(const oracle_lexer* l, int q, int c, int* emit) {
  return lex_step(to_lexer(l), q, c, emit);
}

// Lex `len` bytes from state q.  Writes emitted terminals (skips omitted) to
// out (capacity cap); with flush != 0 the final lexeme is flushed.  Returns the
// number of terminals, -1 if the lexer dies, -2 if cap is too small.
// *final_state receives the state after the bytes (before any flush).
int oracle_lex_bytes(const oracle_lexer* l, int q, const uint8_t* bytes, int len, int flush, int32_t* out, int cap,
                     int* final_state) {
  Lexer L = to_lexer(l);
  int n = 0;
  for (int i = 0; i < len; ++i) {
    int o;
    q = lex_step(L, q, bytes[i], &o);
    if (q == kDead) return -1;
    if (o >= 0) {
      if (n >= cap) return -2;
      out[n++] = o;
    }
  }
  if (final_state) *final_state = q;
  if (flush) {
    int o;
    if (!lex_flush(L, q, &o)) return -1;
    if (o >= 0) {
      if (n >= cap) return -2;
      out[n++] = o;
    }
  }
  return n;
}

// Memo table, token-major, 16-byte canonical entries:
//   [0..1] next state (u16, 0xFFFF = dead)   [2] number of emissions (skips included)
//   [3] emission mask (bit j: an emission happened on reading byte j of the token)
//   [4..11] emitted labels in order (terminal id, 0xFF = skip), unused = 0
//   [12..15] zero.  A dead entry is all zero except next = 0xFFFF.
// Returns 0, or -1 if a token is longer than 8 bytes.
int oracle_memo(const oracle_lexer* l, const oracle_vocab* v, uint8_t* out) {
  Lexer L = to_lexer(l);
  Vocab V = to_vocab(v);
  for (int t = 0; t < V.V; ++t) {
    int len = V.offs[t + 1] - V.offs[t];
    if (len > 8 || len < 1) return -1;
    for (int q0 = 0; q0 < L.Q; ++q0) {
      uint8_t* e = out + ((size_t)t * L.Q + q0) * 16;
      std::memset(e, 0, 16);
      int q = q0, n = 0, mask = 0;
      uint8_t labels[8] = {0};
      bool dead = false;
      for (int j = 0; j < len; ++j) {
        int o;
        q = lex_step(L, q, V.bytes[V.offs[t] + j], &o);
        if (q == kDead) { dead = true; break; }
        if (o != kNone) {
          labels[n++] = (o == kSkip) ? 0xFF : (uint8_t)o;
          mask |= 1 << j;
        }
      }
      if (dead) {
        e[0] = 0xFF;
        e[1] = 0xFF;
        continue;
      }
      e[0] = (uint8_t)(q & 0xFF);
      e[1] = (uint8_t)(q >> 8);
      e[2] = (uint8_t)n;
      e[3] = (uint8_t)mask;
      std::memcpy(e + 4, labels, 8);
    }
  }
  return 0;
}

// Valid(x): 1, 0, or -3 (DFA state limit exceeded).  x: n tokens, -1 = mask.
int oracle_valid(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* x, int n) {
  std::vector<int32_t> xs(x, x + n);
  return valid_seq(to_lexer(l), to_grammar(g), to_vocab(v), xs);
}

// Relaxed(x): 1, 0, or -3.
int oracle_cover(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* x, int n) {
  std::vector<int32_t> xs(x, x + n);
  return relaxed_seq(to_lexer(l), to_grammar(g), to_vocab(v), xs);
}

// Witness of x (failure recovery, Sec. 4): returns 1 and writes the bytes of
// each maximal masked run of x, in order, to out (gap_len[j] bytes for run j,
// *num_gaps runs); 0 when x is not valid; -3 on a construction limit; -2 when
// out or gap_len is too small.
int oracle_witness(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* x, int n,
                   uint8_t* out, int cap, int32_t* gap_len, int max_gaps, int32_t* num_gaps) {
  std::vector<int32_t> xs(x, x + n);
  std::vector<std::vector<uint8_t>> gaps;
  const int r = witness_seq(to_lexer(l), to_grammar(g), to_vocab(v), xs, gaps);
  *num_gaps = (int32_t)gaps.size();
  if (r != 1) return r;
  if ((int)gaps.size() > max_gaps) return -2;
  int k = 0;
  for (size_t j = 0; j < gaps.size(); ++j) {
    if (k + (int)gaps[j].size() > cap) return -2;
    std::memcpy(out + k, gaps[j].data(), gaps[j].size());
    gap_len[j] = (int32_t)gaps[j].size();
    k += (int)gaps[j].size();
  }
  return 1;
}

// Valid of a byte string with no masks: 1 when its greedy lexing is defined
// and in L(G) (Sec. 3 with M(x) empty), 0 otherwise, -3 on a limit.
int oracle_valid_text(const oracle_lexer* l, const oracle_grammar* g, const uint8_t* text, int len) {
  std::vector<int> slots(text, text + len);
  CharNFA A;
  build_char_nfa(to_lexer(l), slots, A);
  DFA D;
  if (!determinize(A, g->num_terminals, D, 4000000)) return -3;
  if (D.start >= 0) minimize(D);
  GrammarView gv(to_grammar(g));
  return earley_accepts(gv, D) ? 1 : 0;
}

// The prior pipeline ("Con.") on candidates, as oracle_validate_batch:
// verdict[c] in {0, 1} (2 malformed); ms[0..2] = summed lexing-automaton,
// determinise-and-minimise and intersection times over all candidates (the
// threads' times added).  Returns 0, or -3 on the DFA limit.
int oracle_con_validate_batch(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v,
                              const int32_t* seqs, int B, int n, const int32_t* cseq, const int32_t* cpos,
                              const int32_t* ctok, int C, uint8_t* verdict, double* ms, int nthreads) {
  const Lexer L = to_lexer(l);
  const Grammar G = to_grammar(g);
  const Vocab V = to_vocab(v);
  std::atomic<int> err{0};
  std::vector<std::array<double, 3>> part(C, std::array<double, 3>{0, 0, 0});
  run_parallel(C, nthreads, [&](int c) {
    const int b = cseq[c], i = cpos[c], t = ctok[c];
    if (b < 0 || b >= B || i < 0 || i >= n || t < 0 || t >= V.V || seqs[(size_t)b * n + i] >= 0) {
      verdict[c] = 2;
      return;
    }
    std::vector<int32_t> x(seqs + (size_t)b * n, seqs + (size_t)(b + 1) * n);
    x[i] = t;
    const int r = con_check(L, G, V, x, part[c].data());
    if (r < 0) err = r;
    verdict[c] = (uint8_t)(r < 0 ? 2 : r);
  });
  for (int k = 0; k < 3; ++k) ms[k] = 0;
  for (auto& pc : part)
    for (int k = 0; k < 3; ++k) ms[k] += pc[k];
  return err.load();
}

// Number of states of x's completion DFA after Hopcroft minimisation (the
// prior pipeline's), -3 on blow-up.
int oracle_con_dfa_states(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* x,
                          int n) {
  std::vector<int32_t> xs(x, x + n);
  int st = 0;
  const int r = con_check(to_lexer(l), to_grammar(g), to_vocab(v), xs, nullptr, &st);
  return r < 0 ? r : st;
}

// Number of states of the minimal completion DFA of x (diagnostics), -3 on blow-up.
int oracle_dfa_states(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* x, int n) {
  DFA D;
  if (!completion_dfa(to_lexer(l), to_grammar(g), to_vocab(v), x, n, D)) return -3;
  return D.start < 0 ? 0 : D.states();
}

// Candidate verdicts: verdict[c] = Valid(x_{seq[c]} + {(pos[c], tok[c])}) in {0,1};
// 2 when the candidate is malformed (sequence or position out of range, the
// position not masked, the token out of range).  Returns 0, or -3 on blow-up.
int oracle_validate_batch(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* seqs,
                          int B, int n, const int32_t* cseq, const int32_t* cpos, const int32_t* ctok, int C,
                          uint8_t* verdict, int nthreads) {
  Lexer L = to_lexer(l);
  Grammar G = to_grammar(g);
  Vocab V = to_vocab(v);
  std::atomic<int> err{0};
  run_parallel(C, nthreads, [&](int c) {
    int b = cseq[c], i = cpos[c], t = ctok[c];
    if (b < 0 || b >= B || i < 0 || i >= n || t < 0 || t >= V.V || seqs[(size_t)b * n + i] >= 0) {
      verdict[c] = 2;
      return;
    }
    std::vector<int32_t> x(seqs + (size_t)b * n, seqs + (size_t)(b + 1) * n);
    x[i] = t;
    int r = valid_seq(L, G, V, x);
    if (r < 0) {
      err = r;
      verdict[c] = 2;
    } else {
      verdict[c] = (uint8_t)r;
    }
  });
  return err.load();
}

// Alg. 4 per sequence over the candidates with verdict 1.  selected[c] = 1 for
// the returned subset.  stats (optional, 2 longs): cover and exact calls.
// Returns 0; -4 if two verdict-1 candidates of one sequence share a position
// or a confidence is NaN (that sequence selects nothing); -3 on blow-up.
int oracle_select(const oracle_lexer* l, const oracle_grammar* g, const oracle_vocab* v, const int32_t* seqs, int B,
                  int n, const int32_t* cseq, const int32_t* cpos, const int32_t* ctok, const float* conf,
                  const uint8_t* verdict, int C, uint8_t* selected, long* stats, int nthreads) {
  Lexer L = to_lexer(l);
  Grammar G = to_grammar(g);
  Vocab V = to_vocab(v);
  std::memset(selected, 0, C);
  std::atomic<int> err{0};
  std::atomic<long> ncover{0}, nexact{0};
  run_parallel(B, nthreads, [&](int b) {
    std::vector<Cand> cs;
    for (int c = 0; c < C; ++c)
      if (cseq[c] == b && verdict[c] == 1) cs.push_back(Cand{c, cpos[c], ctok[c], conf[c]});
    std::set<int> positions;
    for (const Cand& c : cs) {
      if (c.conf != c.conf || !positions.insert(c.pos).second) {
        err = -4;
        return;
      }
    }
    std::stable_sort(cs.begin(), cs.end(), [](const Cand& a, const Cand& b2) { return a.conf > b2.conf; });
    std::vector<int32_t> x(seqs + (size_t)b * n, seqs + (size_t)(b + 1) * n);
    Selector S{L, G, V};
    std::vector<Cand> sel = S.exact_shrink(x, S.relaxed_select(x, cs));
    ncover += S.cover_calls;
    nexact += S.exact_calls;
    if (S.err) {
      err = S.err;
      return;
    }
    for (const Cand& c : sel) selected[c.idx] = 1;
  });
  if (stats) {
    stats[0] = ncover.load();
    stats[1] = nexact.load();
  }
  return err.load();
}

}  // extern "C"
