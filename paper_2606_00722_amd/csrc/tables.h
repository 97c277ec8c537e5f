// Host-side constant tables of the HIP path (built once per context).
#pragma once

#include <cstdint>
#include <string>
#include <vector>

namespace epic {

constexpr int kLabelEps = 63;  // bit 63 of a 64-bit label set = epsilon (skip lexeme)
constexpr int kMaxTerminals = 63;
constexpr int kMaxNonterminals = 64;
constexpr int kMaxStates = 256;
constexpr int kMaxItemWords = 16;  // 512 dotted items
constexpr int kMaxGapClasses = 8;

struct HostTables {
  // sizes
  int Q = 0, T = 0, N = 0, P = 0, NI = 0, W = 0, CW = 0, K = 0, QW = 0, V = 0;
  int start_nt = 0;    // nonterminal index (0..N-1) of the start symbol
  int start_item = 0;  // S' -> . S
  int goal_item = 0;   // S' -> S .
  int max_rhs = 0;
  // lexer
  std::vector<int16_t> trans;     // [Q*256]
  std::vector<int16_t> accept;    // [Q]
  std::vector<uint32_t> ext;      // [Q*QW] states reachable from q without an emission (q included)
  std::vector<uint64_t> flushlab; // [Q] label set of flushing state q (empty = dies)
  // gap automaton, reduced to left-language classes
  std::vector<uint32_t> cls_exit;       // [K*QW] lexer states in which a gap may end inside class k
  std::vector<uint64_t> cls_internal;   // [K*K] labels of edges class k -> class k'
  std::vector<uint64_t> cls_entry;      // [Q*K] labels of edges from an entry lexeme in state q into class k
  std::vector<uint64_t> cls_flush;      // [K]
  // what a masked run derives between its class nodes (independent of the sequence)
  std::vector<uint64_t> gap_nt;   // [K*K] nonterminals deriving a path from class j to class k
  uint64_t gap_eps = 0;           // bit j*K+k: class k reachable from class j by epsilon edges
  std::vector<uint32_t> gap_tm;   // [K*K*W] items that advance from class j to class k
  std::vector<uint32_t> gap_own;  // [K*K*W] entry of the run's origin j at class k
  // grammar (dotted items numbered per production, consecutively)
  std::vector<uint32_t> exp_t;     // [T*W] items whose next symbol is terminal a
  std::vector<uint32_t> exp_n;     // [N*W] items whose next symbol is nonterminal B
  std::vector<uint32_t> pred;      // [N*W] prediction closure of B (nullable nonterminals skipped)
  std::vector<uint32_t> complete;  // [W] items with the dot at the end (augmented item excluded)
  std::vector<int8_t> item_lhs;    // [NI] nonterminal index of the item's production (-1: augmented)
  std::vector<int8_t> next_nt;     // [NI] nonterminal index after the dot (-1: terminal or end)
  std::vector<int8_t> next_sym;    // [NI] symbol after the dot: terminal a, 64 + nonterminal B, -1 at the end
  uint64_t nullable = 0;           // nonterminals deriving the empty string
  std::vector<uint32_t> mn;        // [W] items whose next symbol is a nullable nonterminal
  // nibble-indexed unions: expn_nib[((i*16 + v)*W ..] = union of exp_n[B] over
  // the nonterminals B = 4i + b with bit b of v set; pred_nib likewise for pred
  std::vector<uint32_t> expn_nib;  // [16*16*W]
  std::vector<uint32_t> pred_nib;  // [16*16*W]
  // per item word w and nibble j (bits 4j..4j+3) of it, indexed by the nibble's
  // value: the nonterminals completed by its end items (lhs_nib), and the
  // nonterminals and terminals its items expect (sym_nib: pairs of words)
  std::vector<uint64_t> lhs_nib;  // [W*8*16]
  std::vector<uint64_t> sym_nib;  // [W*8*16*2]
  // the nonterminals and terminals expected by the items of pred_nib's entry
  // (i, v), pairs of words: the symbols a prediction closure expects
  std::vector<uint64_t> predsym_nib;  // [16*16*2]
  std::vector<uint32_t> start_of;  // [N*W] items A -> . gamma
  std::vector<uint32_t> end_of;    // [N*W] items A -> gamma .
  // regular cover: state bit i < 32W is dotted item i (rule position), bit 32W+A is
  // the entry state of nonterminal A, bit 32W+64+A its exit state; cover_cl[s] is
  // the epsilon closure of state s (row of CW words, 32*CW rows)
  std::vector<uint32_t> cover_cl;
  // cover states reachable inside a masked run: gap_cover[((j*K + k)*32*CW + s)*CW ..]
  // is the set of states at class node k reachable from state s at class node j
  // (epsilon moves of the cover and the run's own labelled edges)
  std::vector<uint32_t> gap_cover;
  // witness extraction (failure recovery): terminal strings of what a masked
  // run derives between its class nodes.  A string in wy_pool is a 16-bit
  // length followed by that many terminal ids; offsets are -1 where there is
  // none.  wy_nt[(j*K + k)*N + B]: a string of L(B) labelling a path from class
  // j to class k; wy_own[(j*K + k)*NI + i]: the symbols before the dot of item
  // i (an item of the entry of the run's origin j at class k) derived along a
  // path from class j to class k.
  std::vector<int32_t> wy_nt;
  std::vector<int32_t> wy_own;
  std::vector<uint8_t> wy_pool;
  std::vector<uint32_t> dot0;  // [W] items with the dot at the start of their production
  // vocabulary
  std::vector<uint8_t> vbytes;
  std::vector<int32_t> voffs;
};

// Returns 0 or an epic_status error code; `why` receives a message.
int build_tables(int Q, const int16_t* trans, const int16_t* accept, int T, int N, int start, int P,
                 const int32_t* lhs, const int32_t* roff, const int32_t* rhs, int V, const uint8_t* vbytes,
                 const int32_t* voffs, HostTables& out, std::string& why);

}  // namespace epic
