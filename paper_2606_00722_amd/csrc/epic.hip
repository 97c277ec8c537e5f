// libepic: MI355X (gfx950) implementation of the C ABI in include/epic.h.
//
// Kernels:
//  * lexmemo_kernel  - Alg. 2's lexing memo as a dense table: one thread per
//                      (token, lexer state), token-major so that the rows a
//                      masked gap's exit reads (all states of one token) are
//                      contiguous 16-byte entries.
//  * validate_kernel - one workgroup per candidate (grid-stride over
//                      candidates): the sequence with the candidate applied is
//                      walked into its lexeme graph and recognised by the
//                      Earley engine of walker.inc (Alg. 3).
//  * select_kernel   - one workgroup per sequence runs Alg. 4 with an explicit
//                      stack; every relaxed / exact check is a walk of the
//                      same workgroup (cover policy / Earley policy).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <queue>
#include <random>
#include <string>
#include <vector>

#include "../../include/epic.h"
#include "tables.h"

namespace epic {

// Device helpers are always inlined: a call that takes a kernel argument or a
// work descriptor by reference forces it into per-lane scratch memory, and the
// walks then reload their table pointers from there.
#define EPIC_DEV __device__ inline __attribute__((always_inline))
#define EPIC_INLINE EPIC_DEV
#define EPIC_NOINLINE

__device__ inline int tid() { return (int)threadIdx.x; }
__device__ inline int nthreads() { return (int)blockDim.x; }
__device__ inline void sync() { __syncthreads(); }
__device__ inline uint32_t at_or32(uint32_t* p, uint32_t v) { return atomicOr(p, v); }
__device__ inline uint64_t at_or64(uint64_t* p, uint64_t v) {
  return (uint64_t)atomicOr((unsigned long long*)p, (unsigned long long)v);
}
__device__ inline int at_add32(int32_t* p, int v) { return atomicAdd(p, v); }
__device__ inline unsigned long long at_add64(unsigned long long* p, unsigned long long v) { return atomicAdd(p, v); }
__device__ inline uint32_t at_cas32(uint32_t* p, uint32_t cmp, uint32_t val) { return atomicCAS(p, cmp, val); }
__device__ inline int at_min32(int32_t* p, int v) { return atomicMin(p, v); }
// lane groups: G consecutive lanes of a wavefront (G a power of two <= 64)
__device__ inline uint32_t grp_shfl(uint32_t v, int src, int G) { return (uint32_t)__shfl((int)v, src, G); }
// OR over the group by DPP lane permutations within a row of 16 lanes (swap
// neighbours, swap pairs, mirror each half row, mirror the row); wider groups
// continue with cross-row shuffles
template <int G>
__device__ inline uint32_t grp_or32(uint32_t v) {
  if constexpr (G >= 2) v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0xB1, 0xF, 0xF, false);
  if constexpr (G >= 4) v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x4E, 0xF, 0xF, false);
  if constexpr (G >= 8) v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x141, 0xF, 0xF, false);
  if constexpr (G >= 16) v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x140, 0xF, 0xF, false);
  if constexpr (G >= 32) v |= (uint32_t)__shfl_xor((int)v, 16, 64);
  if constexpr (G >= 64) v |= (uint32_t)__shfl_xor((int)v, 32, 64);
  return v;
}
template <int G>
__device__ inline uint64_t grp_or64(uint64_t v) {
  const uint32_t lo = grp_or32<G>((uint32_t)v), hi = grp_or32<G>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}

#include "walker.inc"

// Threads per walk: two wavefronts per SIMD (512 threads) hide part of the
// memory latency of the chart reads.  Walks of 16-word item sets, whose rows
// are the largest, run on 1024 threads when the launch has no more
// workgroups than the device has CUs (each walk then owns its CU); measured
// best on the C-like workloads of 256 and 1024 tokens.
constexpr int kThreads = 512;
constexpr int kThreadsWide = 1024;
constexpr int kDoneChecks = 64;  // answered checks remembered per sequence by the selection
// Alg. 4 runs several checks per sequence one after another; from this many
// tokens on, each resumes from base walks of the sequence (prefix sharing).
#ifndef EPIC_SHARE_SELECT_LEN
#define EPIC_SHARE_SELECT_LEN 512
#endif
constexpr int kShareSelectLen = EPIC_SHARE_SELECT_LEN;
constexpr int kMemoThreads = 256;

// ------------------------------------------------------------------ memo
#ifndef EPIC_KERNEL_UNIT
__global__ void __launch_bounds__(kMemoThreads) lexmemo_kernel(DevTab tb, uint4* memo) {
  const size_t i = (size_t)blockIdx.x * kMemoThreads + threadIdx.x;
  if (i >= (size_t)tb.V * tb.Q) return;
  const int t = (int)(i / tb.Q), q0 = (int)(i % tb.Q);
  const int beg = tb.voffs[t], len = tb.voffs[t + 1] - beg;  // 1..8 bytes (checked at create)
  // the token's bytes first, all loads in flight together; then the chain of
  // transitions
  int by[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) by[j] = j < len ? tb.vbytes[beg + j] : 0;
  int q = q0;
  uint32_t n = 0, mask = 0, lab_lo = 0, lab_hi = 0;
  bool dead = false;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    if (j >= len) break;
    const int c = by[j];
    const int d = tb.trans[q * 256 + c];
    if (d >= 0) {
      q = d;
      continue;
    }
    const int a = tb.accept[q];
    const int f = tb.trans[c];
    if (a == -1 || f < 0) {
      dead = true;
      break;
    }
    const uint32_t lab = a == -2 ? 0xFFu : (uint32_t)a;
    if (n < 4)
      lab_lo |= lab << (8 * n);
    else
      lab_hi |= lab << (8 * (n - 4));
    mask |= 1u << j;
    ++n;
    q = f;
  }
  uint4 e;
  if (dead) {
    e = make_uint4(0xFFFFu, 0u, 0u, 0u);
  } else {
    e = make_uint4((uint32_t)q | (n << 16) | (mask << 24), lab_lo, lab_hi, 0u);
  }
  memo[i] = e;
}
#endif

// Workspace: nslot chart slots for walks, then base_slots chart slots for
// the base walks of prefix sharing (one per sequence), then one snapshot
// record per base slot.
struct WsArgs {
  char* base;
  size_t slot_bytes;
  size_t off_cnt, off_org, off_sn, off_st, off_bits, off_cov;
  int maxn, maxe, nslot, base_slots, max_seq;
  size_t snap_off, snap_bytes, bseq_off;
};

__device__ inline WgWork slot_work(const WsArgs& a, int slot) {
  char* b = a.base + (size_t)slot * a.slot_bytes;
  WgWork w;
  w.row_off = (int32_t*)b;
  w.row_cnt = (int32_t*)(b + a.off_cnt);
  w.ent_org = (int32_t*)(b + a.off_org);
  w.ent_sn = (uint64_t*)(b + a.off_sn);
  w.ent_st = (uint64_t*)(b + a.off_st);
  w.ent_bits = (uint32_t*)(b + a.off_bits);
  w.cov = (uint32_t*)(b + a.off_cov);
  w.maxn = a.maxn;
  w.maxe = a.maxe;
  w.b_row_off = w.row_off;
  w.b_row_cnt = w.row_cnt;
  w.b_ent_org = w.ent_org;
  w.b_ent_sn = w.ent_sn;
  w.b_ent_st = w.ent_st;
  w.b_ent_bits = w.ent_bits;
  w.b_cov = w.cov;
  w.split_node = 0;
  w.split_ent = 0;
  w.rec = nullptr;
  return w;
}
__device__ inline char* snap_record(const WsArgs& a, int b) { return a.base + a.snap_off + (size_t)b * a.snap_bytes; }

// Resume walk for sequence b at token i0 from its base walk: load the
// snapshot of masked run `run` into LDS (frontier in buffer 0, node
// counters, row mirrors of the shared nodes) and point w's reads of the
// shared prefix at the base chart.
template <int W>
EPIC_INLINE void resume_from_base(Lds<W>& L, const WsArgs& a, int rec, int run, WgWork& w) {
  const WgWork base = slot_work(a, a.nslot + rec);
  const Snapshot* sp = reinterpret_cast<const Snapshot*>(snap_record(a, rec) + kSnapHeader) + run;
  const int t0 = threadIdx.x, NT = blockDim.x;
  const int nn = sp->next_node, ne = sp->ent_cursor, nf = sp->fr_n;
  if (t0 == 0) {
    L.next_node = nn;
    L.ent_cursor = ne;
    L.fr_n[0] = nf;
  }
  for (int i = t0; i < nf * (kQW + 1); i += NT) {
    const int f = i / (kQW + 1), q = i % (kQW + 1);
    if (q == kQW)
      L.fr_node[0][f] = sp->fr_node[f];
    else
      L.fr_set[0][f][q] = sp->fr_set[f][q];
  }
  const int nc = nn < Lds<W>::kNodeCache ? nn : Lds<W>::kNodeCache;
  for (int v = t0; v < nc; v += NT) {
    const int c = base.row_cnt[v];
    L.n_off[v] = base.row_off[v];
    L.n_cnt[v] = (int16_t)((c & kCntMask) | ((c & kOwnFlag) ? 0x8000 : 0));
  }
  w.b_row_off = base.row_off;
  w.b_row_cnt = base.row_cnt;
  w.b_ent_org = base.ent_org;
  w.b_ent_sn = base.ent_sn;
  w.b_ent_st = base.ent_st;
  w.b_ent_bits = base.ent_bits;
  w.b_cov = base.cov;
  w.split_node = nn;
  w.split_ent = ne;
  __syncthreads();
}

// Base walks: sequence b as given, recording its state at every masked run.
// Block b < B walks the Earley graph into base record b; block B + b (when
// launched) walks the cover graph into base record base_slots + b (the two
// graphs can differ: a node lives when its row, or its cover set, is not
// empty).  A record left by an earlier call of the same context (owner tag)
// is reused: the walk state at a masked run depends only on the tokens before
// it, so the walk resumes at the last recorded run that starts at or before
// the first token that differs from the sequence the record was walked on
// (the token there is then walked as the sequence now has it), and a record
// of the very same sequence is kept as it is.
// Base walk number blk (blk < B: the Earley graph of sequence blk; else the
// cover graph of sequence blk - B).  With a nonzero epoch the record's
// progress is published for walks of the same launch (publish_record).
template <int W, int NT>
EPIC_INLINE void base_body(const DevTab& tb, Lds<W>& L, const int32_t* __restrict__ seqs, int B, int n, uint64_t tag,
                           const WsArgs& ws, int blk, uint32_t epoch) {
  const bool cov = blk >= B;
  const int b = cov ? blk - B : blk;
  const int rec = cov ? ws.base_slots + b : b;
  WgWork wk = slot_work(ws, ws.nslot + rec);
  if (threadIdx.x == 0) L.epoch = epoch;
  char* snap = snap_record(ws, rec);
  int32_t* h = reinterpret_cast<int32_t*>(snap);
  int32_t* walked = reinterpret_cast<int32_t*>(ws.base + ws.bseq_off) + (size_t)rec * ws.max_seq;
  if (threadIdx.x == 0) {
    L.sel_bad = 0;
    L.minp = n;   // first token that differs from the recorded sequence
    L.rep_b = -1;  // last recorded run starting before it
  }
  __syncthreads();
  const bool owned = h[2] >= 0 && h[2] <= ws.max_seq && ((uint64_t)(uint32_t)h[4] | ((uint64_t)(uint32_t)h[5] << 32)) == tag &&
                     h[1] >= 0 && h[1] <= ws.max_seq / 2 + 1;
  const int nold = owned ? h[2] : 0;
  for (int k = threadIdx.x; k < n; k += NT) {
    const int x = seqs[(size_t)b * n + k];
    if (x < -1 || x >= tb.V) L.sel_bad = 1;
    L.xtok[k] = x;
    if (k < nold && walked[k] != x) atomicMin(&L.minp, k);
  }
  __syncthreads();
  if (L.sel_bad) {  // an illegal token: no snapshot, candidates report it themselves
    if (threadIdx.x == 0) h[4] = h[5] = 0;  // not reusable
    record_end(L, snap, 2, 0);
    return;
  }
  int d = L.minp < nold ? L.minp : nold;
  if (owned && d == n && nold == n) {  // the record is this sequence's
    publish_record(L, snap, kRecDone | (uint32_t)h[1]);
    return;
  }
  const int runs = owned ? h[1] : 0;
  const Snapshot* sp0 = reinterpret_cast<const Snapshot*>(snap + kSnapHeader);
  for (int r = threadIdx.x; r < runs; r += NT)
    if (sp0[r].start <= d) atomicMax(&L.rep_b, r);
  __syncthreads();
  const int r0 = L.rep_b;
  int i0 = 0;
  if (r0 >= 0) {
    i0 = sp0[r0].start;
    resume_from_base<W>(L, ws, rec, r0, wk);  // the record's own chart up to run r0
  }
  for (int k = threadIdx.x; k < n; k += NT) walked[k] = L.xtok[k];
  if (threadIdx.x == 0) {
    h[2] = n;
    h[4] = (int32_t)(uint32_t)tag;
    h[5] = (int32_t)(uint32_t)(tag >> 32);
  }
  publish_record(L, snap, (uint32_t)(r0 >= 0 ? r0 : 0));  // snapshots before r0 stay as they are
  if (cov)
    walk<W, W, true>(tb, L, wk, n, i0, r0 >= 0, snap, r0 >= 0 ? r0 : 0);
  else
    walk<W, W, false>(tb, L, wk, n, i0, r0 >= 0, snap, r0 >= 0 ? r0 : 0);
}

template <int W, int NT>
__global__ void __launch_bounds__(NT) base_kernel(DevTab tb, const int32_t* __restrict__ seqs, int B, int n,
                                                  uint64_t tag, WsArgs ws) {
  __shared__ Lds<W> L;
  stage_tables<W>(tb, L);
  base_body<W, NT>(tb, L, seqs, B, n, tag, ws, blockIdx.x, 0u);
}

// Thread 0: wait until walk record `snap` holds the snapshot of masked run
// `run` written in launch `epoch`, or is final.  Returns the progress word,
// or 0 when the wait timed out (the caller then walks from the start).
constexpr long long kRecWaitCycles = 4ll << 30;
__device__ inline uint64_t wait_record(const char* snap, uint32_t epoch, int run) {
  const uint64_t* p = reinterpret_cast<const uint64_t*>(snap + 24);
  const long long t_start = (long long)clock64();
  for (;;) {
    // relaxed: an acquire load on every poll would invalidate this XCD's L2
    // under every walk resident there; the caller fences once it returns
    const uint64_t v = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const uint32_t st = (uint32_t)v;
    if ((uint32_t)(v >> 32) == epoch && ((st & kRecDone) || (int)st > run)) return v;
    if ((long long)clock64() - t_start > kRecWaitCycles) return 0;
    __builtin_amdgcn_s_sleep(8);
  }
}

// ------------------------------------------------------------------ validate
// Candidate walks blk, blk + nblk, ... in walk slot blk.  With SHARE each
// resumes from its sequence's base walk; with a nonzero epoch those base
// walks run in the same launch and the walk first waits for its snapshot.
template <int W, int NT, bool SHARE>
EPIC_INLINE void validate_body(const DevTab& tb, Lds<W>& L, const int32_t* __restrict__ seqs, int B, int n,
                               const int32_t* __restrict__ cseq, const int32_t* __restrict__ cpos,
                               const int32_t* __restrict__ ctok, int C, uint8_t* __restrict__ verdict,
                               const WsArgs& ws, int blk, int nblk, uint32_t epoch) {
  const WgWork wk = slot_work(ws, blk);
  for (int c = blk; c < C; c += nblk) {
    const int b = cseq[c], i = cpos[c], t = ctok[c];
    const bool bad = b < 0 || b >= B || i < 0 || i >= n || t < 0 || t >= tb.V || seqs[(size_t)b * n + i] >= 0;
    if (bad) {
      if (threadIdx.x == 0) {
        verdict[c] = 2;
        atomicOr(tb.dev_err, (uint32_t)EPIC_DEV_BAD_CANDIDATE);
      }
      continue;
    }
    if (threadIdx.x == 0) L.sel_bad = 0;
    __syncthreads();
    for (int k = threadIdx.x; k < n; k += (int)blockDim.x) {
      const int x = k == i ? t : seqs[(size_t)b * n + k];
      if (x < -1 || x >= tb.V) L.sel_bad = 1;
      L.xtok[k] = x;
    }
    __syncthreads();
    if (L.sel_bad) {  // a token of the sequence is out of range
      if (threadIdx.x == 0) {
        verdict[c] = 2;
        atomicOr(tb.dev_err, (uint32_t)EPIC_DEV_BAD_CANDIDATE);
      }
      __syncthreads();
      continue;
    }
    int r;
    if (SHARE) {
      // the masked run of x_b holding position i: its start p0 and ordinal
      if (threadIdx.x == 0) {
        L.minp = -1;  // last fixed position before i
        L.rep_b = 0;  // masked runs starting before p0
      }
      __syncthreads();
      for (int k = threadIdx.x; k < i; k += NT)
        if (L.xtok[k] >= 0) atomicMax(&L.minp, k);
      __syncthreads();
      const int p0 = L.minp + 1;
      for (int k = threadIdx.x; k < p0; k += NT)
        if (L.xtok[k] < 0 && (k == 0 || L.xtok[k - 1] >= 0)) atomicAdd(&L.rep_b, 1);
      __syncthreads();
      const int run = L.rep_b;
      const int32_t* h = reinterpret_cast<const int32_t*>(snap_record(ws, b));
      int ready = 1;  // 1: the record is final; 2: snapshot `run` is written; 0: not waited for in time
      if (epoch) {
        __syncthreads();
        if (threadIdx.x == 0) {
          const uint64_t v = wait_record(snap_record(ws, b), epoch, run);
          L.result = v == 0 ? 0 : (((uint32_t)v & kRecDone) ? 1 : 2);
        }
        __syncthreads();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        ready = L.result;
      }
      const int status = ready == 1 ? h[0] : 0, runs = ready == 1 ? h[1] : run + 1;
      if (ready == 0) {
        r = walk<W, W, false>(tb, L, wk, n);
      } else if (run < runs) {
        WgWork wr = wk;
        resume_from_base<W>(L, ws, b, run, wr);
        r = walk<W, W, false>(tb, L, wr, n, p0, true);
      } else {
        r = status == 1 ? 0 : -1;  // the shared prefix died, or overflowed
        if (threadIdx.x == 0 && r < 0) L.overflow = kOvEntries;
      }
    } else {
      r = walk<W, W, false>(tb, L, wk, n);
    }
    if (threadIdx.x == 0) {
      verdict[c] = (uint8_t)(r < 0 ? 2 : r);
      if (r < 0) atomicOr(tb.dev_err, (uint32_t)EPIC_DEV_CAPACITY | (1u << (8 + (L.overflow & 15))));
    }
    __syncthreads();
  }
}

template <int W, int NT, bool SHARE>
__global__ void __launch_bounds__(NT) validate_kernel(DevTab tb, const int32_t* __restrict__ seqs, int B,
                                                            int n, const int32_t* __restrict__ cseq,
                                                            const int32_t* __restrict__ cpos,
                                                            const int32_t* __restrict__ ctok, int C,
                                                            uint8_t* __restrict__ verdict, WsArgs ws) {
  __shared__ Lds<W> L;
  stage_tables<W>(tb, L);
  validate_body<W, NT, SHARE>(tb, L, seqs, B, n, cseq, cpos, ctok, C, verdict, ws, blockIdx.x, gridDim.x, 0u);
}

// Base walks and the candidate walks that resume from them in one launch:
// workgroups 0 .. gb-1 are the base walks (as base_kernel), the others the
// candidate walks (as validate_kernel), each of which waits until the base
// walk of its sequence has written the snapshot it resumes from, so that
// candidate walks overlap the rest of the base walks.  Base walks have the
// lowest workgroup numbers and wait on nothing, so they are dispatched first
// and finish; a candidate walk that is not released in time walks from the
// start instead.  The base walks' work counts apart (base_work).
template <int W, int NT>
__global__ void __launch_bounds__(NT) base_validate_kernel(DevTab tb, const int32_t* __restrict__ seqs, int B, int n,
                                                           uint64_t tag, int gb, const int32_t* __restrict__ cseq,
                                                           const int32_t* __restrict__ cpos,
                                                           const int32_t* __restrict__ ctok, int C,
                                                           uint8_t* __restrict__ verdict, WsArgs ws, uint32_t epoch,
                                                           unsigned long long* base_work) {
  __shared__ Lds<W> L;
  stage_tables<W>(tb, L);
  if ((int)blockIdx.x < gb) {
    if (threadIdx.x == 0) L.work_to = base_work;
    base_body<W, NT>(tb, L, seqs, B, n, tag, ws, blockIdx.x, epoch);
  } else {
    validate_body<W, NT, true>(tb, L, seqs, B, n, cseq, cpos, ctok, C, verdict, ws, blockIdx.x - gb,
                               gridDim.x - gb, epoch);
  }
}

// ------------------------------------------------------------------ select
// Alg. 4 as a stack machine run by thread 0; checks are walks by the whole
// workgroup.  Subsets are bit masks over the confidence-sorted candidates.
// The host runs the same machine to plan speculated checks.
enum : int { kRS = 0, kES = 1, kTop = 2 };
enum : int { kReqNone = 0, kReqCover = 1, kReqExact = 2, kReqDone = 3 };

struct Frame {
  int type, stage;
  uint64_t A, S, t1;
};

__host__ __device__ inline int popc64(uint64_t x) { return __builtin_popcountll(x); }

__host__ __device__ inline void split_halves(uint64_t S, uint64_t& lo, uint64_t& hi) {
  int cnt = popc64(S), h = (cnt + 1) / 2;  // ceil(|S|/2) on the high-confidence side
  lo = 0;
  uint64_t s = S;
  for (int i = 0; i < h; ++i) {
    uint64_t bit = s & (~s + 1);
    lo |= bit;
    s &= s - 1;
  }
  hi = S & ~lo;
}

// ExactShrink(x, RelaxedSelect(x, C)) over the m sorted candidates: advance()
// runs until the machine asks a check (req = kReqCover or kReqExact on
// `mask`) or finishes (req = kReqDone, the selection in final_B); the caller
// puts the check's outcome in res before the next advance().
struct Alg4 {
  Frame stack[96];  // depth <= 2 + 3 * log2(64) frames
  int sp, req, res;
  uint64_t mask, ret_val, final_B;
};

__host__ __device__ inline void alg4_start(Alg4& a, int m) {
  a.stack[0] = Frame{kTop, 0, 0, m >= 64 ? ~0ull : ((1ull << m) - 1), 0};
  a.sp = 1;
  a.req = kReqNone;
  a.res = 0;
  a.mask = 0;
  a.ret_val = 0;
  a.final_B = 0;
}

__host__ __device__ inline void alg4_advance(Alg4& a) {
  a.req = kReqNone;
  while (a.req == kReqNone) {
    if (a.sp == 0 || a.sp >= 95) {  // >= 95 cannot happen for <= 64 candidates
      a.req = kReqDone;
      break;
    }
    Frame& f = a.stack[a.sp - 1];
    if (f.type == kTop) {
      if (f.stage == 0) {
        f.stage = 1;
        a.stack[a.sp++] = Frame{kRS, 0, 0, f.S, 0};
      } else if (f.stage == 1) {
        f.stage = 2;
        a.stack[a.sp++] = Frame{kES, 0, 0, a.ret_val, 0};
      } else {
        a.final_B = a.ret_val;
        --a.sp;
      }
      continue;
    }
    const bool is_rs = f.type == kRS;
    if (f.stage == 0) {
      if (popc64(f.S) <= 1) {
        a.ret_val = 0;
        --a.sp;
        continue;
      }
      f.stage = 1;
      a.req = is_rs ? kReqCover : kReqExact;
      a.mask = f.A | f.S;
      break;
    }
    if (f.stage == 1) {
      if (a.res) {
        a.ret_val = f.S;
        --a.sp;
        continue;
      }
      uint64_t lo, hi;
      split_halves(f.S, lo, hi);
      f.stage = 2;
      a.stack[a.sp++] = Frame{is_rs ? kRS : kES, 0, f.A, lo, 0};
      continue;
    }
    if (f.stage == 2) {
      uint64_t lo, hi;
      split_halves(f.S, lo, hi);
      f.t1 = a.ret_val;  // B_L (RelaxedSelect) or B'_L (ExactShrink)
      f.stage = 3;
      a.stack[a.sp++] = Frame{kRS, 0, f.A | f.t1, hi, 0};
      continue;
    }
    if (f.stage == 3) {
      if (is_rs) {
        a.ret_val = f.t1 | a.ret_val;
        --a.sp;
        continue;
      }
      f.stage = 4;  // B'_R = ret_val; now ExactShrink(x + B'_L, B'_R)
      a.stack[a.sp++] = Frame{kES, 0, f.A | f.t1, a.ret_val, 0};
      continue;
    }
    // ExactShrink stage 4: B''_R = ret_val
    a.ret_val = f.t1 | a.ret_val;
    --a.sp;
  }
}

// Answered checks: Alg. 4 asks some again (after an exact check fails and a
// half passes, the next RelaxedSelect and ExactShrink repeat the cover and
// exact checks of the whole set).  The selection remembers the first
// kDoneChecks answers of a sequence; a check found here is not walked.
__host__ __device__ inline int done_find(const uint64_t* msk, const int* val, int n, uint64_t m, int kind) {
  int hit = -1;
  for (int k = 0; k < n; ++k)
    if (msk[k] == m && (val[k] & 2) == kind) hit = val[k] & 1;
  return hit;
}

// The outcome of a check (cover or exact, on subset m) that an answered
// check (cover2, subset m2, outcome r2) decides, else -1.  A masked run
// reads any bytes, so filling more positions only shrinks the character
// language of x: checks are monotone in the subset (a pass carries to its
// subsets, a failure to its supersets); and the cover's language contains
// L(G), so an exact pass implies a cover pass and a cover failure an exact
// failure.
__host__ __device__ inline int implied_outcome(bool cover, uint64_t m, bool cover2, uint64_t m2, int r2) {
  if (r2 == 1 && (m & ~m2) == 0 && (cover2 == cover || !cover2)) return 1;
  if (r2 == 0 && (m2 & ~m) == 0 && (cover2 == cover || cover2)) return 0;
  return -1;
}

// Replays the machine from its start along a path of outcomes (bit i: the
// outcome of the i-th check not found in the answered checks) until the
// check at depth d; false when the machine finishes first.  On true, a.req
// and a.mask are that check.
__host__ __device__ inline bool alg4_replay(Alg4& a, int m, uint64_t path, int d, uint64_t* dmsk, int* dval, int& dn) {
  alg4_start(a, m);
  dn = 0;
  int depth = 0;
  for (int guard = 0; guard < 1 << 16; ++guard) {
    alg4_advance(a);
    if (a.req == kReqDone) return false;
    const int kind = a.req == kReqCover ? 2 : 0;
    const int hit = done_find(dmsk, dval, dn, a.mask, kind);
    if (hit >= 0) {
      a.res = hit;
      continue;
    }
    if (depth == d) return true;
    const int r = (int)((path >> depth) & 1);
    ++depth;
    if (dn < kDoneChecks) {
      dmsk[dn] = a.mask;
      dval[dn] = r | kind;
      ++dn;
    }
    a.res = r;
  }
  return false;
}

// The candidates Alg. 4 selects from for sequence b: its verdict-1
// candidates, sorted by descending confidence with ties to the lower
// candidate index, into L.sel_idx/pos/tok/conf (L.sel_n of them).  Clears
// the sequence's selected flags when `selected` is given.  Returns L.sel_bad:
// 0 ok, 1 repeated position or NaN confidence, 2 more than 64 candidates,
// 3 a verdict-1 candidate or a sequence token that is not legal.
template <int W>
EPIC_DEV int select_setup(const DevTab& tb, Lds<W>& L, const int32_t* __restrict__ seqs, int n,
                            const int32_t* __restrict__ cseq, const int32_t* __restrict__ cpos,
                            const int32_t* __restrict__ ctok, const float* __restrict__ conf,
                            const uint8_t* __restrict__ verdict, int C, int b, uint8_t* __restrict__ selected) {
  if (threadIdx.x == 0) {
    L.sel_n = 0;
    L.sel_bad = 0;
  }
  __syncthreads();
  for (int c = threadIdx.x; c < C; c += (int)blockDim.x) {
    if (cseq[c] != b) continue;
    if (selected) selected[c] = 0;
    if (verdict[c] != 1) continue;
    const int i = cpos[c], t = ctok[c];
    if (i < 0 || i >= n || t < 0 || t >= tb.V || seqs[(size_t)b * n + i] >= 0) {
      L.sel_bad = 3;  // a verdict-1 candidate that is not a legal update
      continue;
    }
    int j = atomicAdd(&L.sel_n, 1);
    if (j < 64) L.sel_idx[j] = c;
  }
  for (int k = threadIdx.x; k < n; k += (int)blockDim.x) {
    const int x = seqs[(size_t)b * n + k];
    if (x < -1 || x >= tb.V) L.sel_bad = 3;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int m = L.sel_n;
    if (L.sel_bad) {
    } else if (m > 64) {
      L.sel_bad = 2;
    } else {
      // order by candidate index, then stable sort by descending confidence
      for (int i = 1; i < m; ++i)
        for (int j = i; j > 0 && L.sel_idx[j - 1] > L.sel_idx[j]; --j) {
          int tmp = L.sel_idx[j];
          L.sel_idx[j] = L.sel_idx[j - 1];
          L.sel_idx[j - 1] = tmp;
        }
      for (int i = 0; i < m; ++i) {
        int c = L.sel_idx[i];
        L.sel_pos[i] = cpos[c];
        L.sel_tok[i] = ctok[c];
        L.sel_conf[i] = conf[c];
        if (!(L.sel_conf[i] == L.sel_conf[i])) L.sel_bad = 1;
        for (int j = 0; j < i; ++j)
          if (L.sel_pos[j] == L.sel_pos[i]) L.sel_bad = 1;
      }
      for (int i = 1; i < m; ++i)
        for (int j = i; j > 0 && L.sel_conf[j - 1] < L.sel_conf[j]; --j) {
          int ti = L.sel_idx[j];
          L.sel_idx[j] = L.sel_idx[j - 1];
          L.sel_idx[j - 1] = ti;
          ti = L.sel_pos[j];
          L.sel_pos[j] = L.sel_pos[j - 1];
          L.sel_pos[j - 1] = ti;
          ti = L.sel_tok[j];
          L.sel_tok[j] = L.sel_tok[j - 1];
          L.sel_tok[j - 1] = ti;
          float tf = L.sel_conf[j];
          L.sel_conf[j] = L.sel_conf[j - 1];
          L.sel_conf[j - 1] = tf;
        }
    }
  }
  __syncthreads();
  return L.sel_bad;
}

// Sequence b with the sorted candidates in mask applied, into L.xtok.
template <int W>
EPIC_DEV void select_apply(Lds<W>& L, const int32_t* __restrict__ seqs, int n, int b, uint64_t msk) {
  for (int k = threadIdx.x; k < n; k += (int)blockDim.x) L.xtok[k] = seqs[(size_t)b * n + k];
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int i = 0; i < L.sel_n; ++i)
      if ((msk >> i) & 1) L.xtok[L.sel_pos[i]] = L.sel_tok[i];
  }
  __syncthreads();
}

// One check of Alg. 4 for sequence b: the walk of x_b with the sorted
// candidates in msk applied (relaxed: cover graph; exact: Earley graph).
// With `share`, the walk resumes from the sequence's base walk at the masked
// run holding the subset's lowest position: x_b and x_b + S agree before it.
template <int W, bool COVER, bool SHARE>
EPIC_INLINE int select_walk_body(const DevTab& tb, Lds<W>& L, const WgWork& wk, const WsArgs& ws,
                           const int32_t* __restrict__ seqs, int n, int b, uint64_t msk) {
  select_apply<W>(L, seqs, n, b, msk);
  if constexpr (!SHARE) {
    return walk<W, W, COVER>(tb, L, wk, n);
  } else {
  WgWork wr = wk;
  int p0 = 0;
  bool resume = false;
  {
    if (threadIdx.x == 0) {
      int pmin = n;
      for (int i = 0; i < L.sel_n; ++i)
        if (((msk >> i) & 1) && L.sel_pos[i] < pmin) pmin = L.sel_pos[i];
      L.minp = -1;  // last fixed position before pmin
      L.rep_b = 0;  // masked runs starting before the run of pmin
      L.result = pmin;
    }
    __syncthreads();
    const int pmin = L.result;
    for (int k = threadIdx.x; k < pmin; k += blockDim.x)
      if (L.xtok[k] >= 0) atomicMax(&L.minp, k);
    __syncthreads();
    p0 = L.minp + 1;
    for (int k = threadIdx.x; k < p0; k += blockDim.x)
      if (L.xtok[k] < 0 && (k == 0 || L.xtok[k - 1] >= 0)) atomicAdd(&L.rep_b, 1);
    __syncthreads();
    const int run = L.rep_b, rec = COVER ? ws.base_slots + b : b;
    const int32_t* h = reinterpret_cast<const int32_t*>(snap_record(ws, rec));
    const int status = h[0], runs = h[1];
    if (run >= runs) {
      if (status == 1) return 0;  // the shared prefix died
      if (threadIdx.x == 0) L.overflow = kOvEntries;
      __syncthreads();
      return -1;
    }
    resume_from_base<W>(L, ws, rec, run, wr);
    resume = true;
  }
  return walk<W, W, COVER>(tb, L, wr, n, resume ? p0 : 0, resume);
  }
}

// A check walk kept as a function of its own for 16-word item sets in the
// selection.  It measured faster than the inlined walk although its call
// frame costs more per-lane scratch: at 1024 threads per workgroup (128
// registers per lane), where the inlined walk spills in its inner loops,
// 29.7 against 31.7 ms of C-like selection per 256-token step; at 512
// threads, on checks resumed from base walks, 4.12 against 4.44 ms per
// 1024-token step.  Narrower item sets, and the sequential fallback, inline
// it.
// It takes the walk slot's index, not its descriptor: a descriptor passed by
// reference would live in per-lane scratch, and the walk would read its
// pointers from there.
template <int W, bool COVER, bool SHARE>
__device__ __attribute__((noinline)) int select_walk_call(const DevTab& tb, Lds<W>& L, int slot, const WsArgs& ws,
                                                          const int32_t* __restrict__ seqs, int n, int b,
                                                          uint64_t msk) {
  const WgWork wk = slot_work(ws, slot);
  return select_walk_body<W, COVER, SHARE>(tb, L, wk, ws, seqs, n, b, msk);
}

// `wk` is the workgroup's own walk slot (slot_work(ws, blockIdx.x)).
template <int W, bool COVER, bool SHARE, bool CALL = (W >= 16)>
EPIC_INLINE int select_walk(const DevTab& tb, Lds<W>& L, const WgWork& wk, const WsArgs& ws,
                                  const int32_t* __restrict__ seqs, int n, int b, uint64_t msk) {
  if constexpr (CALL)
    return select_walk_call<W, COVER, SHARE>(tb, L, (int)blockIdx.x, ws, seqs, n, b, msk);
  else
    return select_walk_body<W, COVER, SHARE>(tb, L, wk, ws, seqs, n, b, msk);
}

// Speculated checks.  The machine's next check depends only on the number m
// of candidates and on the outcomes of the checks it has made, so its checks
// form one binary decision tree per m.  A node is a path of outcomes: those
// of the checks before it that were not found among the answered checks.
// The root, the relaxed check of all candidates, is the selection's own
// first walk.  For every m the host explores the tree below the root by
// decreasing estimated probability (outcomes taken as independent, a
// relaxed check passing with probability 0.75, an exact one with 0.9) and
// lists the first kPlan distinct checks (kind and subset) it meets, each
// with a level: twice the negative base-2 logarithm of that probability,
// rounded down.  Helper workgroups take (sequence, planned check) pairs
// level by level, sequence by sequence within a level, walk the check and
// publish the result in a state word (0 not started, 1 running, 3 nothing to
// do, 4 + the outcome when done).  When the selection needs a check, it
// looks it up among the planned checks of its m: it takes a result that is
// done, waits for one that is running (its helper is resident and finishes
// on its own), and otherwise walks the check itself.  A check's outcome
// depends only on its kind and subset, so the plan decides only which
// checks run early, not any result.
constexpr int kPlan = 64;        // planned nodes (state slots) per sequence
constexpr int kPlanLevels = 32;  // levels of the helper order
// (the C-like 1024-token trajectory's checks pass at 0.62 and 0.79; these
// higher estimates, which reach deeper along passing paths, measured 1.5-2 %
// faster there and 1.5 % slower on C-like 256-token steps)
constexpr double kPlanPassRelaxed = 0.75, kPlanPassExact = 0.9;
// Plan table (int32 words): level starts [65][kPlanLevels + 1] (the checks
// of m at level l are kPlan*m + start[l] .. start[l+1]-1; start[kPlanLevels]
// is their count), then the checks [65][kPlan] as {kind (kReqCover or
// kReqExact), level, subset low word, subset high word}.
constexpr int kPlanNodeWord = 65 * (kPlanLevels + 1);
constexpr int kPlanWords = kPlanNodeWord + 65 * kPlan * 4;
// Helpers per sequence at most (a launch also leaves every workgroup a CU
// and a chart slot): with the planned checks, 15 helpers at 16 sequences
// measured faster than 5 (C-like 256-token selection 25.8 -> 23.9 ms).
constexpr int kSpecHelpers = 31;
// Speculation block of a selection launch over B sequences (int32 words):
// state [B*kPlan], consulted flag [B*kPlan], then the work counters of each
// speculated check's walk (uint64 [B*kPlan][6]).  A state word carries the
// result too (kSpecDone + outcome, or kSpecDone + 2 when the walk ran out of
// capacity), so that publishing and reading it need no cache write-back or
// invalidation: one relaxed agent-scope store, relaxed polls.
enum : int { kSpecIdle = 0, kSpecRunning = 1, kSpecNone = 3, kSpecDone = 4 };
constexpr int spec_work_word(int B) { return (2 * B * kPlan + 1) & ~1; }
constexpr int spec_words(int B) { return spec_work_word(B) + 2 * 6 * B * kPlan; }
constexpr long long kSpecWaitCycles = 4ll << 30;  // give up waiting on a helper after this many clocks
constexpr int kSpecSeqs = 128;  // sequences a launch with helpers may hold

// Helpers per sequence at most: its first kPlanUse planned nodes.
constexpr int kPlanUse = 64;

// Helper pairs at level l of a sequence with m candidates.
__device__ inline int plan_level_count(const int32_t* plan, int m, int l) {
  if (m < 2 || m > 64) return 0;
  const int32_t* st = plan + m * (kPlanLevels + 1);
  const int a = st[l] < kPlanUse ? st[l] : kPlanUse, b = st[l + 1] < kPlanUse ? st[l + 1] : kPlanUse;
  return b - a;
}

template <int W>
__global__ void spec_clear_kernel(int32_t* __restrict__ state, int count) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < count) state[i] = 0;
}

// After a selection launch: the work of each speculated check's walk goes to
// the selection's counters (`used`: the selection took its result, so the
// walk is one of the algorithm's own checks) or to the speculation's.
template <int W>
__global__ void spec_account_kernel(const int32_t* __restrict__ spec, int B, unsigned long long* used,
                                    unsigned long long* unused) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= B * kPlan) return;
  const unsigned long long* w = reinterpret_cast<const unsigned long long*>(spec + spec_work_word(B)) + (size_t)i * 6;
  if (w[0] == 0) return;
  unsigned long long* to = spec[B * kPlan + i] ? used : unused;
  for (int k = 0; k < 6; ++k) atomicAdd(&to[k], w[k]);
}

template <int W, int NT, bool SHARE>
__global__ void __launch_bounds__(NT) select_kernel(DevTab tb, const int32_t* __restrict__ seqs, int B, int n,
                                                          const int32_t* __restrict__ cseq,
                                                          const int32_t* __restrict__ cpos,
                                                          const int32_t* __restrict__ ctok,
                                                          const float* __restrict__ conf,
                                                          const uint8_t* __restrict__ verdict, int C,
                                                          uint8_t* __restrict__ selected, long long* counts,
                                                          int32_t* __restrict__ spec, WsArgs ws) {
  __shared__ Lds<W> L;
  __shared__ Alg4 M;
  __shared__ uint64_t done_msk[kDoneChecks];
  __shared__ int done_val[kDoneChecks];  // result | (cover ? 2 : 0)
  __shared__ int done_n, done_hit, spec_pick, plan_j, implied;
  const WgWork wk = slot_work(ws, blockIdx.x);
  stage_tables<W>(tb, L);
  int32_t* spec_state = spec;             // [B * kPlan]
  int32_t* spec_used = spec + B * kPlan;  // [B * kPlan]: the selection took the result
  // Workgroups b < B run Alg. 4 for sequence b; the others are helpers, each
  // walking the check of one planned node of a sequence b.  Both reach the
  // walks through the one call site of each check type below.
  const bool helper = (int)blockIdx.x >= B;
  const bool helpers = (int)gridDim.x > B;
  int b = (int)blockIdx.x, hj = 0;
  if (helper) {
    // Helper hi takes the hi-th (sequence, node) pair: by level, then by
    // sequence, then by the node's place in the sequence's plan.  Every
    // helper computes the same order from the verdicts: the valid candidates
    // per sequence, then a prefix sum over the (level, sequence) cells.  The
    // walk's origin hash is free until the first walk, which clears it.
    int* spec_m = reinterpret_cast<int*>(L.hash);  // [B]: valid candidates
    static_assert(kSpecSeqs <= kHash, "helper counts fit in the origin hash");
    const int hi = (int)blockIdx.x - B;
    for (int k = threadIdx.x; k < B; k += (int)blockDim.x) spec_m[k] = 0;
    if (threadIdx.x == 0) spec_pick = -1;
    __syncthreads();
    for (int c = threadIdx.x; c < C; c += (int)blockDim.x) {
      const int cb = cseq[c];
      if (cb >= 0 && cb < B && verdict[c] == 1) atomicAdd(&spec_m[cb], 1);
    }
    __syncthreads();
    const int ncell = kPlanLevels * B, per = (ncell + (int)blockDim.x - 1) / (int)blockDim.x;
    const int c0 = (int)threadIdx.x * per, c1 = c0 + per < ncell ? c0 + per : ncell;
    int sum = 0;
    for (int c = c0; c < c1; ++c) sum += plan_level_count(tb.plan, spec_m[c % B], c / B);
    int total = 0;
    int acc = block_scan<W>(L, sum, &total);
    if (hi >= acc && hi < acc + sum)
      for (int c = c0; c < c1; ++c) {
        const int bb = c % B, lvl = c / B, k = plan_level_count(tb.plan, spec_m[bb], lvl);
        if (hi < acc + k) {
          spec_pick = bb * kPlan + tb.plan[spec_m[bb] * (kPlanLevels + 1) + lvl] + (hi - acc);
          break;
        }
        acc += k;
      }
    __syncthreads();
    if (spec_pick < 0) return;  // no planned node left
    b = spec_pick / kPlan;
    hj = spec_pick % kPlan;
  }
  // a speculated check's walk counts its work in its own slot; after the
  // launch it goes to the selection's counters when the selection took the
  // result, else to the speculation's (spec_account_kernel)
  if (helper && threadIdx.x == 0)
    L.work_to = reinterpret_cast<unsigned long long*>(spec + spec_work_word(B)) + (size_t)(b * kPlan + hj) * 6;
  const int bad = select_setup<W>(tb, L, seqs, n, cseq, cpos, ctok, conf, verdict, C, b, helper ? nullptr : selected);
  if (helper) {
    if (threadIdx.x == 0) {
      const int m = L.sel_n;
      bool found = false;
      if (!bad && m >= 2 && m <= 64 && hj < tb.plan[m * (kPlanLevels + 1) + kPlanLevels]) {
        const int32_t* e = tb.plan + kPlanNodeWord + (m * kPlan + hj) * 4;
        M.req = e[0];
        M.mask = (uint64_t)(uint32_t)e[2] | ((uint64_t)(uint32_t)e[3] << 32);
        found = true;
      }
      plan_j = found ? 1 : 0;
      __hip_atomic_store(&spec_state[b * kPlan + hj], found ? kSpecRunning : kSpecNone, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!plan_j) return;
  } else if (threadIdx.x == 0) {
    if (L.sel_bad)
      atomicOr(tb.dev_err, L.sel_bad == 2   ? (uint32_t)EPIC_DEV_CAPACITY
                           : L.sel_bad == 3 ? (uint32_t)EPIC_DEV_BAD_CANDIDATE
                                            : (uint32_t)EPIC_DEV_BAD_SELECT);
    done_n = 0;
    alg4_start(M, L.sel_n);
  }
  __syncthreads();
  if (!helper && L.sel_bad) return;
  long long ncover = 0, nexact = 0;
  bool failed = false;
  for (int step = 0; step < 1 << 20; ++step) {
    int req;
    uint64_t msk;
    int r = -1;
    if (helper) {
      req = M.req;
      msk = M.mask;
    } else {
      if (threadIdx.x == 0) alg4_advance(M);
      __syncthreads();
      req = M.req;
      if (req == kReqDone) break;
      msk = M.mask;
      if (req == kReqCover)
        ++ncover;
      else
        ++nexact;
      const int kind = req == kReqCover ? 2 : 0;
      if (threadIdx.x == 0) {
        done_hit = done_find(done_msk, done_val, done_n, msk, kind);
        plan_j = -1;
        implied = -1;
      }
      __syncthreads();
      r = done_hit;
      if (r < 0 && step > 0) {
        // decided by an answered check: the selection's own, or a helper's
        // finished one (all such answers agree)
        const bool cov = req == kReqCover;
        for (int k = threadIdx.x; k < done_n; k += (int)blockDim.x) {
          const int o = implied_outcome(cov, msk, (done_val[k] & 2) != 0, done_msk[k], done_val[k] & 1);
          if (o >= 0) implied = o;
        }
        if (helpers) {
          const int m = L.sel_n;
          const int cnt = tb.plan[m * (kPlanLevels + 1) + kPlanLevels];
          for (int j = threadIdx.x; j < cnt; j += (int)blockDim.x) {
            const int st = __hip_atomic_load(&spec_state[b * kPlan + j], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (st != kSpecDone && st != kSpecDone + 1) continue;
            const int32_t* e = tb.plan + kPlanNodeWord + (m * kPlan + j) * 4;
            const uint64_t sub = (uint64_t)(uint32_t)e[2] | ((uint64_t)(uint32_t)e[3] << 32);
            const int o = implied_outcome(cov, msk, e[0] == kReqCover, sub, st - kSpecDone);
            if (o >= 0) {
              implied = o;
              spec_used[b * kPlan + j] = 1;
            }
          }
        }
        __syncthreads();
        r = implied;
      }
      if (r < 0 && helpers && step > 0) {
        // this check among the planned ones, if it is there (a running one:
        // waited for; finished ones were looked at above)
        const int m = L.sel_n;
        const int cnt = tb.plan[m * (kPlanLevels + 1) + kPlanLevels];
        for (int j = threadIdx.x; j < cnt; j += (int)blockDim.x) {
          const int32_t* e = tb.plan + kPlanNodeWord + (m * kPlan + j) * 4;
          const uint64_t sub = (uint64_t)(uint32_t)e[2] | ((uint64_t)(uint32_t)e[3] << 32);
          if (e[0] == req && sub == msk) plan_j = j;
        }
        __syncthreads();
        const int q = plan_j;
        if (q >= 0 && threadIdx.x == 0) {
          int res = -1;
          const long long t_start = (long long)clock64();
          while ((long long)clock64() - t_start < kSpecWaitCycles) {
            const int st = __hip_atomic_load(&spec_state[b * kPlan + q], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (st == kSpecDone || st == kSpecDone + 1) res = st - kSpecDone;
            if (st != kSpecRunning) break;
            __builtin_amdgcn_s_sleep(8);
          }
          if (res >= 0) spec_used[b * kPlan + q] = 1;
          L.sel_res = res;
        }
        if (q >= 0) {
          __syncthreads();
          r = L.sel_res;
        }
      }
    }
    const bool fresh = done_hit < 0;
    if (r < 0)
      r = req == kReqCover ? select_walk<W, true, SHARE>(tb, L, wk, ws, seqs, n, b, msk)
                           : select_walk<W, false, SHARE>(tb, L, wk, ws, seqs, n, b, msk);
    if (helper) {
      if (threadIdx.x == 0) {
        // capacity (r < 0): the selection walks the check again and reports it
        __hip_atomic_store(&spec_state[b * kPlan + hj], kSpecDone + (r < 0 ? 2 : r), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
      return;
    }
    if (r < 0) {
      failed = true;
      break;
    }
    if (threadIdx.x == 0) {
      M.res = r;
      if (fresh && done_n < kDoneChecks) {
        done_msk[done_n] = msk;
        done_val[done_n] = r | (req == kReqCover ? 2 : 0);
        ++done_n;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    if (counts) {
      atomicAdd((unsigned long long*)&counts[0], (unsigned long long)ncover);
      atomicAdd((unsigned long long*)&counts[1], (unsigned long long)nexact);
    }
    if (failed) {
      atomicOr(tb.dev_err, (uint32_t)EPIC_DEV_CAPACITY | (1u << (8 + (L.overflow & 15))));
    } else {
      for (int i = 0; i < L.sel_n; ++i)
        if ((M.final_B >> i) & 1) selected[L.sel_idx[i]] = 1;
    }
  }
}

// ------------------------------------------------------------------ fallback
// The sequential fallback that follows the relaxed batch in EPIC decoding
// (Alg. 1 in App. C.1, and the paragraph after it): with the
// selected set B committed, the remaining candidates of sequence b are taken
// by descending confidence (ties to the lower candidate index) and each is
// committed when x + (everything committed so far) + c is valid, until
// num_commit[b] - |B| more are committed or the candidates run out.  Only
// verdict-1 candidates are walked: filling masked positions only shrinks the
// character language of x (a masked run reads any bytes), so a candidate
// invalid on x stays invalid on every later x.  One workgroup per sequence;
// the checks are the selection's exact walks (with SHARE, resumed from the
// sequence's base walk at the masked run of the lowest committed position).
// Helpers of the fallback: workgroups from nprim on each check one
// remaining candidate i of one sequence against the selected set alone
// (x + B + c_i), concurrently with the loops.  Checks are monotone in the
// subset (a masked run reads any bytes), so when the loop reaches i with
// committed set K (B within K): a failure there decides that x + K + c_i
// fails too, and while K is still B a pass is the loop's very check.  Helper
// hi takes the hi-th (j, sequence) pair, j-th remaining candidate first;
// results go to state words as the selection's (4 + outcome when done).
template <int W, int NT, bool SHARE>
__global__ void __launch_bounds__(NT) fallback_kernel(DevTab tb, const int32_t* __restrict__ seqs, int B, int n,
                                                      const int32_t* __restrict__ cseq,
                                                      const int32_t* __restrict__ cpos,
                                                      const int32_t* __restrict__ ctok,
                                                      const float* __restrict__ conf,
                                                      const uint8_t* __restrict__ verdict,
                                                      const uint8_t* __restrict__ selected,
                                                      const int32_t* __restrict__ num_commit, int C,
                                                      uint8_t* __restrict__ accepted, WsArgs ws, int nprim,
                                                      int32_t* __restrict__ spec) {
  __shared__ Lds<W> L;
  __shared__ uint64_t kept;  // sorted candidates committed: B, then the accepted ones
  __shared__ int need, pick, decided;
  const WgWork wk = slot_work(ws, blockIdx.x);
  stage_tables<W>(tb, L);
  const bool helpers = (int)gridDim.x > nprim;
  if ((int)blockIdx.x >= nprim) {
    // remaining (valid, not selected) candidates per sequence, then the
    // hi-th pair over the (j, sequence) cells; the origin hash is free
    // until the walk, which clears it
    int* rem = reinterpret_cast<int*>(L.hash);  // [B]
    const int hi = (int)blockIdx.x - nprim;
    for (int k = threadIdx.x; k < B; k += (int)blockDim.x) rem[k] = 0;
    if (threadIdx.x == 0) pick = -1;
    __syncthreads();
    for (int c = threadIdx.x; c < C; c += (int)blockDim.x) {
      const int cb = cseq[c];
      if (cb >= 0 && cb < B && verdict[c] == 1 && !selected[c]) atomicAdd(&rem[cb], 1);
    }
    __syncthreads();
    const int ncell = 64 * B, per = (ncell + (int)blockDim.x - 1) / (int)blockDim.x;
    const int c0 = (int)threadIdx.x * per, c1 = c0 + per < ncell ? c0 + per : ncell;
    int sum = 0;
    for (int c = c0; c < c1; ++c) sum += c / B < rem[c % B];
    int total = 0;
    int acc = block_scan<W>(L, sum, &total);
    if (hi >= acc && hi < acc + sum)
      for (int c = c0; c < c1; ++c) {
        if (!(c / B < rem[c % B])) continue;
        if (acc == hi) {
          pick = c;
          break;
        }
        ++acc;
      }
    __syncthreads();
    if (pick < 0) return;
    const int b = pick % B, j = pick / B;
    select_setup<W>(tb, L, seqs, n, cseq, cpos, ctok, conf, verdict, C, b, nullptr);
    if (threadIdx.x == 0) {
      // the j-th remaining candidate in confidence order, and B
      uint64_t k0 = 0;
      int i = -1, r = 0;
      for (int q = 0; q < L.sel_n; ++q) {
        if (selected[L.sel_idx[q]])
          k0 |= 1ull << q;
        else if (r++ == j)
          i = q;
      }
      kept = k0;
      pick = L.sel_bad || i < 0 ? -1 : i;
      if (pick >= 0)
        __hip_atomic_store(&spec[b * kPlan + pick], kSpecRunning, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    const int i = pick;
    if (i < 0) return;
    const int r = select_walk<W, false, SHARE, false>(tb, L, wk, ws, seqs, n, b, kept | (1ull << i));
    if (threadIdx.x == 0)
      __hip_atomic_store(&spec[b * kPlan + i], kSpecDone + (r < 0 ? 2 : r), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
    return;
  }
  for (int b = blockIdx.x; b < B; b += nprim) {
    // sorts b's verdict-1 candidates and clears accepted[] of all of b's
    select_setup<W>(tb, L, seqs, n, cseq, cpos, ctok, conf, verdict, C, b, accepted);
    uint64_t k0 = 0;  // B
    if (threadIdx.x == 0) {
      if (L.sel_bad)
        atomicOr(tb.dev_err, L.sel_bad == 2   ? (uint32_t)EPIC_DEV_CAPACITY
                             : L.sel_bad == 3 ? (uint32_t)EPIC_DEV_BAD_CANDIDATE
                                              : (uint32_t)EPIC_DEV_BAD_SELECT);
      uint64_t k = 0;
      for (int i = 0; i < L.sel_n; ++i)
        if (selected[L.sel_idx[i]]) k |= 1ull << i;
      kept = k;
      need = num_commit[b] - __popcll(k);
    }
    __syncthreads();
    k0 = kept;
    if (!L.sel_bad) {
      for (int i = 0; i < L.sel_n && need > 0; ++i) {
        if ((kept >> i) & 1) continue;
        int r = -1;
        if (helpers) {
          // a helper's check of x + B + c_i: a failure decides; a pass decides
          // while nothing beyond B is committed (then it is this check, and
          // a running one is waited for)
          if (threadIdx.x == 0) {
            const bool same = kept == k0;
            int res = -1;
            const long long t_start = (long long)clock64();
            while ((long long)clock64() - t_start < kSpecWaitCycles) {
              const int st = __hip_atomic_load(&spec[b * kPlan + i], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
              if (st == kSpecDone || (st == kSpecDone + 1 && same)) res = st - kSpecDone;
              if (st != kSpecRunning || !same) break;
              __builtin_amdgcn_s_sleep(8);
            }
            decided = res;
          }
          __syncthreads();
          r = decided;
        }
        if (r < 0) r = select_walk<W, false, SHARE, false>(tb, L, wk, ws, seqs, n, b, kept | (1ull << i));
        if (r < 0) {
          if (threadIdx.x == 0)
            atomicOr(tb.dev_err, (uint32_t)EPIC_DEV_CAPACITY | (1u << (8 + (L.overflow & 15))));
          break;
        }
        if (threadIdx.x == 0 && r) {
          kept |= 1ull << i;
          --need;
          accepted[L.sel_idx[i]] = 1;
        }
        __syncthreads();
      }
    }
    __syncthreads();
  }
}

#include "witness.inc"

}  // namespace epic

// ==================================================================== C ABI
using namespace epic;

// Kernel kinds for the diagnostics: each kind's walks add to a work-counter
// set of its own, and with timing on each launch is bracketed by HIP events.
// kKSelectHelp: the work counters of the speculated checks whose results the
// selection did not take (walked by its helper workgroups besides the
// algorithm's own checks); it has no launches of its own (its time is the
// selection's).  kKSpecClear times the speculation bookkeeping: the state
// clear before a selection launch and the work accounting after it.
enum : int { kKLexmemo = 0, kKBase, kKValidate, kKSelect, kKFallback, kKSpecClear, kKSelectHelp, kKernelKinds };
constexpr int kWorkCounters = 6;   // counters per set (see epic_ctx_work_counters)
constexpr size_t kWorkOff = 64;    // byte offset of the counter sets in the error block
constexpr size_t kErrBlock = 1024; // bytes of the error / counter block

struct epic_ctx {
  HostTables H;
  int max_batch = 0, max_seq = 0, max_cands = 0;
  int maxn = 0, maxe = 0, nslot = 0;
  size_t slot_bytes = 0, ws_bytes = 0;
  size_t off_cnt = 0, off_org = 0, off_sn = 0, off_st = 0, off_bits = 0, off_cov = 0;
  void* d_tables = nullptr;
  uint4* d_memo = nullptr;
  uint32_t* d_err = nullptr;
  DevTab tab{};
  bool memo_built = false;
  int device = 0;
  int num_cus = 256;
  int base_slots = 0;
  size_t off_snap = 0, snap_bytes = 0, off_spec = 0, off_bseq = 0;
  uint64_t tag = 0;  // owner tag of the base records this context writes
  uint32_t epoch = 0;  // launches of base and candidate walks together (walk-record progress words)
  void* scratch = nullptr;  // this device's static scratch (epic_validate_batch_noalloc)
  // witness workspace layout, per sequence (epic_witness)
  int wit_lds_proofs = kWitLdsSlots / 2;  // proofs indexed in LDS by the back-trace
  int wit_lds_vis = kWitVisLds;           // visited-set words of a masked run kept in LDS
  size_t wit_stride = 0, wit_rec = 0, wit_mark = 0, wit_stack = 0, wit_w = 0, wit_recs = 0, wit_vis = 0;
  size_t wit_proof = 0, wit_pindex = 0, wit_sys = 0;
  int wit_ecap = 0;
  // diagnostics: per-kernel HIP-event timing (epic_ctx_set_timing)
  bool timing = false;
  struct Pending {
    int kid;
    hipEvent_t a, b;
  };
  std::vector<Pending> pending;
  double kernel_ms[kKernelKinds] = {};
  int64_t kernel_launches[kKernelKinds] = {};
};

namespace {

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

template <class T>
size_t place(std::vector<char>& blob, const std::vector<T>& v) {
  size_t off = align256(blob.size());
  blob.resize(off + std::max<size_t>(v.size() * sizeof(T), 1));
  if (!v.empty()) std::memcpy(blob.data() + off, v.data(), v.size() * sizeof(T));
  return off;
}

// The selection's speculation plan: for m = 2..64 candidates, the distinct
// checks met exploring the machine's decision tree below the root by
// decreasing estimated probability, best first (a node's children are its
// check's two outcomes), in the layout of kPlanWords.  The same for every
// context.
const std::vector<int32_t>& speculation_plan() {
  static const std::vector<int32_t> plan = [] {
    std::vector<int32_t> pl(kPlanWords, 0);
    struct Node {
      double nl;  // -log2 of the estimated probability
      uint64_t path;
      int depth;
    };
    auto later = [](const Node& x, const Node& y) {
      if (x.nl != y.nl) return x.nl > y.nl;
      if (x.depth != y.depth) return x.depth > y.depth;
      return x.path > y.path;
    };
    std::unique_ptr<Alg4> a(new Alg4);
    uint64_t dmsk[kDoneChecks];
    int dval[kDoneChecks];
    for (int m = 2; m <= 64; ++m) {
      std::priority_queue<Node, std::vector<Node>, decltype(later)> heap(later);
      heap.push(Node{0.0, 0, 0});
      std::vector<Node> nodes;
      std::vector<std::pair<int, uint64_t>> checks;  // (kind, subset) of nodes[j]
      for (int pops = 0; !heap.empty() && (int)nodes.size() < kPlan && pops < 1 << 16; ++pops) {
        const Node x = heap.top();
        heap.pop();
        int dn = 0;
        if (!alg4_replay(*a, m, x.path, x.depth, dmsk, dval, dn)) continue;  // the machine finishes first
        const std::pair<int, uint64_t> ck(a->req, a->mask);
        if (x.depth > 0 && std::find(checks.begin(), checks.end(), ck) == checks.end()) {
          nodes.push_back(x);
          checks.push_back(ck);
        }
        if (x.depth >= 63) continue;
        const double p = a->req == kReqCover ? kPlanPassRelaxed : kPlanPassExact;
        heap.push(Node{x.nl - std::log2(p), x.path | (1ull << x.depth), x.depth + 1});
        heap.push(Node{x.nl - std::log2(1.0 - p), x.path, x.depth + 1});
      }
      int32_t* st = pl.data() + m * (kPlanLevels + 1);
      int32_t* nd = pl.data() + kPlanNodeWord + m * kPlan * 4;
      int l = 0;
      for (int j = 0; j < (int)nodes.size(); ++j) {
        const int lvl = std::min(kPlanLevels - 1, (int)(2.0 * nodes[j].nl));
        while (l <= lvl) st[l++] = j;
        nd[4 * j] = checks[j].first;
        nd[4 * j + 1] = lvl;
        nd[4 * j + 2] = (int32_t)(uint32_t)checks[j].second;
        nd[4 * j + 3] = (int32_t)(uint32_t)(checks[j].second >> 32);
      }
      while (l <= kPlanLevels) st[l++] = (int)nodes.size();
    }
    return pl;
  }();
  return plan;
}

epic_status upload(epic_ctx* c) {
  const HostTables& H = c->H;
  std::vector<char> blob;
  size_t o_trans = place(blob, H.trans), o_accept = place(blob, H.accept), o_ext = place(blob, H.ext),
         o_flush = place(blob, H.flushlab), o_cexit = place(blob, H.cls_exit), o_cint = place(blob, H.cls_internal),
         o_centry = place(blob, H.cls_entry), o_cflush = place(blob, H.cls_flush), o_expt = place(blob, H.exp_t),
         o_expn = place(blob, H.exp_n), o_pred = place(blob, H.pred), o_comp = place(blob, H.complete),
         o_lhs = place(blob, H.item_lhs), o_nsym = place(blob, H.next_sym), o_mn = place(blob, H.mn),
         o_gtm = place(blob, H.gap_tm), o_gown = place(blob, H.gap_own), o_ccl = place(blob, H.cover_cl),
         o_enib = place(blob, H.expn_nib), o_pnib = place(blob, H.pred_nib), o_gcov = place(blob, H.gap_cover),
         o_lnib = place(blob, H.lhs_nib), o_snib = place(blob, H.sym_nib), o_psnib = place(blob, H.predsym_nib), o_plan = place(blob, speculation_plan()),
         o_vb = place(blob, H.vbytes), o_vo = place(blob, H.voffs), o_endof = place(blob, H.end_of),
         o_dot0 = place(blob, H.dot0), o_wynt = place(blob, H.wy_nt), o_wyown = place(blob, H.wy_own),
         o_wypool = place(blob, H.wy_pool);
  {
    // owner tag of the walk records this context writes: FNV-1a over every
    // constant table (the memo is a function of them) and the workspace
    // layout, mixed with a per-process random value and a per-context count,
    // so that records of another context, another process or other tables
    // never match
    uint64_t h = 1469598103934665603ull;
    auto mix = [&h](const void* p, size_t n) {
      const unsigned char* b = (const unsigned char*)p;
      for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
    };
    mix(blob.data(), blob.size());
    const size_t layout[] = {c->slot_bytes, (size_t)c->maxn, (size_t)c->maxe, (size_t)c->nslot,
                             (size_t)c->base_slots, (size_t)c->max_seq, c->snap_bytes, c->off_snap, c->off_bseq};
    mix(layout, sizeof(layout));
    static const uint64_t nonce = ((uint64_t)std::random_device{}() << 32) ^ std::random_device{}();
    static std::atomic<uint64_t> counter{1};
    c->tag = h ^ (nonce + 0x9E3779B97F4A7C15ull * counter.fetch_add(1));
    if (c->tag == 0) c->tag = 1;  // a zeroed header never matches
  }
  if (hipMalloc(&c->d_tables, blob.size()) != hipSuccess) return EPIC_ERR_HIP;
  if (hipMemcpy(c->d_tables, blob.data(), blob.size(), hipMemcpyHostToDevice) != hipSuccess) return EPIC_ERR_HIP;
  if (hipMalloc((void**)&c->d_memo, (size_t)H.V * H.Q * sizeof(uint4)) != hipSuccess) return EPIC_ERR_HIP;
  if (hipMalloc((void**)&c->d_err, kErrBlock) != hipSuccess) return EPIC_ERR_HIP;
  if (hipMemset(c->d_err, 0, kErrBlock) != hipSuccess) return EPIC_ERR_HIP;
  char* d = (char*)c->d_tables;
  DevTab& t = c->tab;
  t.Q = H.Q;
  t.T = H.T;
  t.N = H.N;
  t.NI = H.NI;
  t.W = H.W;
  t.CW = H.CW;
  t.K = H.K;
  t.QW = H.QW;
  t.V = H.V;
  t.start_nt = H.start_nt;
  t.start_item = H.start_item;
  t.goal_item = H.goal_item;
  t.trans = (const int16_t*)(d + o_trans);
  t.accept = (const int16_t*)(d + o_accept);
  t.ext = (const uint32_t*)(d + o_ext);
  t.flushlab = (const uint64_t*)(d + o_flush);
  t.cls_exit = (const uint32_t*)(d + o_cexit);
  t.cls_internal = (const uint64_t*)(d + o_cint);
  t.cls_entry = (const uint64_t*)(d + o_centry);
  t.cls_flush = (const uint64_t*)(d + o_cflush);
  t.exp_t = (const uint32_t*)(d + o_expt);
  t.exp_n = (const uint32_t*)(d + o_expn);
  t.pred = (const uint32_t*)(d + o_pred);
  t.complete = (const uint32_t*)(d + o_comp);
  t.item_lhs = (const int8_t*)(d + o_lhs);
  t.next_sym = (const int8_t*)(d + o_nsym);
  t.mn = (const uint32_t*)(d + o_mn);
  t.gap_tm = (const uint32_t*)(d + o_gtm);
  t.gap_own = (const uint32_t*)(d + o_gown);
  t.gap_eps = H.gap_eps;
  t.expn_nib = (const uint32_t*)(d + o_enib);
  t.pred_nib = (const uint32_t*)(d + o_pnib);
  t.gap_cover = (const uint32_t*)(d + o_gcov);
  t.lhs_nib = (const uint64_t*)(d + o_lnib);
  t.sym_nib = (const uint64_t*)(d + o_snib);
  t.predsym_nib = (const uint64_t*)(d + o_psnib);
  t.plan = (const int32_t*)(d + o_plan);
  t.cover_cl = (const uint32_t*)(d + o_ccl);
  t.vbytes = (const uint8_t*)(d + o_vb);
  t.voffs = (const int32_t*)(d + o_vo);
  t.end_of = (const uint32_t*)(d + o_endof);
  t.dot0 = (const uint32_t*)(d + o_dot0);
  t.nullable = H.nullable;
  t.wy_nt = (const int32_t*)(d + o_wynt);
  t.wy_own = (const int32_t*)(d + o_wyown);
  t.wy_pool = (const uint8_t*)(d + o_wypool);
  t.memo = c->d_memo;
  t.dev_err = c->d_err;
  t.work = (unsigned long long*)((char*)c->d_err + kWorkOff);
  return EPIC_OK;
}

WsArgs ws_args(const epic_ctx* c, void* ws) {
  WsArgs a;
  a.base = (char*)ws;
  a.slot_bytes = c->slot_bytes;
  a.off_cnt = c->off_cnt;
  a.off_org = c->off_org;
  a.off_sn = c->off_sn;
  a.off_st = c->off_st;
  a.off_bits = c->off_bits;
  a.off_cov = c->off_cov;
  a.maxn = c->maxn;
  a.maxe = c->maxe;
  a.nslot = c->nslot;
  a.base_slots = c->base_slots;
  a.max_seq = c->max_seq;
  a.bseq_off = c->off_bseq;
  a.snap_off = c->off_snap;
  a.snap_bytes = c->snap_bytes;
  return a;
}

constexpr int kWitFrames = 1 << 15;    // back-trace stack
constexpr int kWitTerminals = 1 << 15; // terminals of a witness
constexpr int kWitRecords = 1 << 20;   // byte-search records
constexpr int kWitProofs = 1 << 18;    // stored proofs of the back-trace
constexpr int kWitProofSlots = 1 << 19;
constexpr int kWitSystems = 1 << 12;   // masked-run systems ranked by the back-trace
constexpr int kWitVisWords = 1 << 15;  // byte-search visited set (bits: lexer states x window)
constexpr int kWitSteps = 1 << 22;     // back-trace steps

WitArgs wit_args(const epic_ctx* c, void* wws) {
  WitArgs a;
  a.base = (char*)wws;
  a.stride = c->wit_stride;
  a.off_rec = c->wit_rec;
  a.off_mark = c->wit_mark;
  a.off_stack = c->wit_stack;
  a.off_w = c->wit_w;
  a.off_recs = c->wit_recs;
  a.off_vis = c->wit_vis;
  a.off_proof = c->wit_proof;
  a.off_pindex = c->wit_pindex;
  a.off_sys = c->wit_sys;
  a.syscap = kWitSystems;
  a.pcap = kWitProofs;
  a.pslots = kWitProofSlots;
  a.ecap = c->wit_ecap;
  a.scap = kWitFrames;
  a.wcap = kWitTerminals;
  a.rcap = kWitRecords;
  a.vwords = kWitVisWords;
  a.steps = kWitSteps;
  a.lproofs = c->wit_lds_proofs;
  a.lvis = c->wit_lds_vis;
  return a;
}

// The context's tables with the work counters of kernel kind kid.
DevTab tab_for(const epic_ctx* c, int kid) {
  DevTab t = c->tab;
  t.work = (unsigned long long*)((char*)c->d_err + kWorkOff) + (size_t)kid * 8;
  return t;
}

// Brackets one kernel launch with HIP events on its stream when the
// context's timing diagnostics are on.
struct KernelTimer {
  epic_ctx* c;
  int kid;
  hipStream_t s;
  hipEvent_t a = nullptr, b = nullptr;
  KernelTimer(epic_ctx* c_, int kid_, hipStream_t s_) : c(c_), kid(kid_), s(s_) {
    if (!c->timing) return;
    if (hipEventCreate(&a) != hipSuccess || hipEventCreate(&b) != hipSuccess) {
      a = b = nullptr;
      return;
    }
    (void)hipEventRecord(a, s);
  }
  ~KernelTimer() {
    if (!a) return;
    (void)hipEventRecord(b, s);
    c->pending.push_back({kid, a, b});
  }
};

}  // namespace

// Launchers of one item width.  Each width's kernels are compiled in a unit of
// their own (epic_w<W>.hip defines EPIC_KERNEL_UNIT as W and includes this
// file), so the widths build in parallel; this unit holds the C ABI.
template <int W>
struct ValidateLaunch {
  static epic_status run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs, const int32_t* cp,
                         const int32_t* ct, int C, uint8_t* verdict, void* ws, hipStream_t stream);
};

template <int W>
struct SelectLaunch {
  static epic_status run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs, const int32_t* cp,
                         const int32_t* ct, const float* conf, const uint8_t* verdict, int C, uint8_t* sel,
                         int64_t* counts, void* ws, hipStream_t stream);
};

// Candidate walks only (no prefix sharing), in the slots of a caller-given
// region: the launch of epic_validate_batch_noalloc.
template <int W>
struct ValidatePlainLaunch {
  static epic_status run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs, const int32_t* cp,
                         const int32_t* ct, int C, uint8_t* verdict, void* region, int nslot, hipStream_t stream);
};

template <int W>
struct FallbackLaunch {
  static epic_status run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs, const int32_t* cp,
                         const int32_t* ct, const float* conf, const uint8_t* verdict, const uint8_t* sel,
                         const int32_t* num_commit, int C, uint8_t* accepted, void* ws, hipStream_t stream);
};

template <int W>
struct WitnessLaunch {
  static epic_status run(epic_ctx* c, const int32_t* seqs, int B, int n, uint8_t* bytes, int bytes_per_seq,
                         int32_t* gap_len, int max_gaps, int32_t* status, void* wws, void* ws, hipStream_t stream);
};

#ifdef EPIC_KERNEL_UNIT
// Base walks of sequences 0..B-1 (gb = B: Earley graphs; 2B: also the cover
// graphs).
template <int W>
void launch_base(epic_ctx* c, const int32_t* seqs, int B, int n, int gb, const WsArgs& wa, hipStream_t stream) {
  KernelTimer kt(c, kKBase, stream);
  const DevTab tb = tab_for(c, kKBase);
  // 512 threads also for 16-word item sets: at 1024 (128 registers per
  // lane) the walk spills and measured slower (C-like 1024-token base walks
  // 1.13 against 1.10 ms)
  hipLaunchKernelGGL((base_kernel<W, kThreads>), dim3(gb), dim3(kThreads), 0, stream, tb, seqs, B, n, c->tag, wa);
}

// Whether validation walks the base walks of both graphs and the selection's
// checks resume from them: for long sequences, and whenever those 2B walks
// fit beside the candidate walks on the CUs (shorter sequences: JSON-like
// 128-token steps 12.7K -> 13.3K checks/s, SMILES-like 256-token 9.85K ->
// 10.2K; where they do not fit, C-like 256-token steps lost 30 %).
static bool share_both(const epic_ctx* c, int B, int n, int C) {
  return B <= c->base_slots && (n >= kShareSelectLen || std::min(C, c->nslot) + 2 * B <= c->num_cus);
}

template <int W>
epic_status ValidateLaunch<W>::run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs,
                                   const int32_t* cp, const int32_t* ct, int C, uint8_t* verdict, void* ws,
                                   hipStream_t stream) {
  int grid = std::min(C, c->nslot);
  const WsArgs wa = ws_args(c, ws);
  const DevTab tb = tab_for(c, kKValidate);
  const bool both = share_both(c, B, n, C);
  if ((grid > c->num_cus || both) && B <= c->base_slots) {
    // more walks than CUs, or base walks of both graphs (share_both): the
    // chart up to each candidate's masked run is its sequence's, walked by a
    // base walk (prefix sharing; the cover graphs' base walks are the
    // selection's)
    // base walks and candidate walks in one launch (base_validate_kernel)
    const int gb = both ? 2 * B : B;
    if (++c->epoch == 0) ++c->epoch;  // 0 means "no waiting"
    KernelTimer kt(c, kKValidate, stream);
    hipLaunchKernelGGL((base_validate_kernel<W, kThreads>), dim3(gb + grid), dim3(kThreads), 0, stream, tb, seqs, B,
                       n, c->tag, gb, cs, cp, ct, C, verdict, wa, c->epoch, tab_for(c, kKBase).work);
  } else if (W >= 16 && grid <= c->num_cus) {
    KernelTimer kt(c, kKValidate, stream);
    hipLaunchKernelGGL((validate_kernel<W, kThreadsWide, false>), dim3(grid), dim3(kThreadsWide), 0, stream, tb, seqs,
                       B, n, cs, cp, ct, C, verdict, wa);
  } else {
    KernelTimer kt(c, kKValidate, stream);
    hipLaunchKernelGGL((validate_kernel<W, kThreads, false>), dim3(grid), dim3(kThreads), 0, stream, tb, seqs, B, n, cs,
                       cp, ct, C, verdict, wa);
  }
  return hipGetLastError() == hipSuccess ? EPIC_OK : EPIC_ERR_HIP;
}

template <int W>
epic_status SelectLaunch<W>::run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs,
                                 const int32_t* cp, const int32_t* ct, const float* conf, const uint8_t* verdict,
                                 int C, uint8_t* sel, int64_t* counts, void* ws, hipStream_t stream) {
  int32_t* spec = (int32_t*)((char*)ws + c->off_spec);
  // B selection workgroups, then up to kSpecHelpers helpers per sequence,
  // as many as leave every workgroup a CU and a chart slot
  const int nh = std::min({kSpecHelpers, c->num_cus / B - 1, c->nslot / B - 1});
  const int grid = nh >= 1 && B <= kSpecSeqs ? B * (nh + 1) : B;
  const WsArgs wa = ws_args(c, ws);
  // Alg. 4's checks resume from base walks of both graphs when validation
  // walked them (share_both); this launch resumes those records, so it walks
  // nothing when the sequences are unchanged since
  const int share = share_both(c, B, n, C);
  if (share) launch_base<W>(c, seqs, B, n, 2 * B, wa, stream);
  {
    KernelTimer kt(c, kKSpecClear, stream);
    hipLaunchKernelGGL(spec_clear_kernel<W>, dim3((spec_words(B) + 255) / 256), dim3(256), 0, stream, spec,
                       spec_words(B));
  }
  // 1024 threads for 16-word item sets when every workgroup has a CU, except
  // for checks resumed from base walks (shorter walks, where 512 threads
  // measured faster: 4.12 against 4.25 ms per C-like 1024-token step)
  const bool wide = W >= 16 && grid <= c->num_cus && !share;
  // The 1024-thread instance of the resumed-check selection is compiled but
  // not launched: the out-of-line check walk that both instances call is then
  // compiled to the 1024-thread register budget (128 per lane), and that code
  // measured faster at 512 threads too (4.13 against 4.40 ms of C-like
  // selection per 1024-token step) than a walk compiled for 512 threads only.
  if constexpr (W >= 16) (void)&select_kernel<W, kThreadsWide, true>;
  const DevTab tb = tab_for(c, kKSelect);
  {
    KernelTimer kt(c, kKSelect, stream);
    if (wide)
      hipLaunchKernelGGL((select_kernel<W, kThreadsWide, false>), dim3(grid), dim3(kThreadsWide), 0, stream, tb, seqs,
                         B, n, cs, cp, ct, conf, verdict, C, sel, (long long*)counts, spec, wa);
    else if (share)
      hipLaunchKernelGGL((select_kernel<W, kThreads, true>), dim3(grid), dim3(kThreads), 0, stream, tb, seqs, B, n,
                         cs, cp, ct, conf, verdict, C, sel, (long long*)counts, spec, wa);
    else
      hipLaunchKernelGGL((select_kernel<W, kThreads, false>), dim3(grid), dim3(kThreads), 0, stream, tb, seqs, B, n,
                         cs, cp, ct, conf, verdict, C, sel, (long long*)counts, spec, wa);
  }
  if (grid > B) {
    KernelTimer kt(c, kKSpecClear, stream);
    hipLaunchKernelGGL(spec_account_kernel<W>, dim3((B * kPlan + 255) / 256), dim3(256), 0, stream, spec, B,
                       tb.work, tab_for(c, kKSelectHelp).work);
  }
  return hipGetLastError() == hipSuccess ? EPIC_OK : EPIC_ERR_HIP;
}

template <int W>
epic_status FallbackLaunch<W>::run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs,
                                   const int32_t* cp, const int32_t* ct, const float* conf, const uint8_t* verdict,
                                   const uint8_t* sel, const int32_t* num_commit, int C, uint8_t* accepted,
                                   void* ws, hipStream_t stream) {
  const int nprim = std::min(B, c->nslot);
  const WsArgs wa = ws_args(c, ws);
  int32_t* spec = (int32_t*)((char*)ws + c->off_spec);
  // helpers as the selection's: as many as leave every workgroup a CU and a
  // chart slot
  const int nh = std::min({kSpecHelpers, c->num_cus / B - 1, c->nslot / B - 1});
  const int grid = nh >= 1 && B <= kSpecSeqs && nprim == B ? B * (nh + 1) : nprim;
  // long sequences: the loop's exact checks resume from the base walks of the
  // Earley graphs, as the selection's do
  const bool share = n >= kShareSelectLen && B <= c->base_slots;
  if (share) launch_base<W>(c, seqs, B, n, B, wa, stream);
  if (grid > nprim) {
    KernelTimer kt(c, kKSpecClear, stream);
    hipLaunchKernelGGL(spec_clear_kernel<W>, dim3((B * kPlan + 255) / 256), dim3(256), 0, stream, spec, B * kPlan);
  }
  KernelTimer kt(c, kKFallback, stream);
  if (share)
    hipLaunchKernelGGL((fallback_kernel<W, kThreads, true>), dim3(grid), dim3(kThreads), 0, stream,
                       tab_for(c, kKFallback), seqs, B, n, cs, cp, ct, conf, verdict, sel, num_commit, C, accepted, wa,
                       nprim, spec);
  else
    hipLaunchKernelGGL((fallback_kernel<W, kThreads, false>), dim3(grid), dim3(kThreads), 0, stream,
                       tab_for(c, kKFallback), seqs, B, n, cs, cp, ct, conf, verdict, sel, num_commit, C, accepted, wa,
                       nprim, spec);
  return hipGetLastError() == hipSuccess ? EPIC_OK : EPIC_ERR_HIP;
}

template <int W>
epic_status ValidatePlainLaunch<W>::run(epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs,
                                        const int32_t* cp, const int32_t* ct, int C, uint8_t* verdict, void* region,
                                        int nslot, hipStream_t stream) {
  WsArgs wa = ws_args(c, region);
  wa.nslot = nslot;  // walk slots 0..nslot-1 only; no base slots or records
  wa.base_slots = 0;
  const int grid = std::min(C, nslot);
  const DevTab tb = tab_for(c, kKValidate);
  if (W >= 16 && grid <= c->num_cus)
    hipLaunchKernelGGL((validate_kernel<W, kThreadsWide, false>), dim3(grid), dim3(kThreadsWide), 0, stream, tb, seqs,
                       B, n, cs, cp, ct, C, verdict, wa);
  else
    hipLaunchKernelGGL((validate_kernel<W, kThreads, false>), dim3(grid), dim3(kThreads), 0, stream, tb, seqs, B, n, cs,
                       cp, ct, C, verdict, wa);
  return hipGetLastError() == hipSuccess ? EPIC_OK : EPIC_ERR_HIP;
}

// Witness extraction: the recording walk of each sequence in chart slot b,
// the back-trace (one wavefront per sequence), the byte search.
template <int W>
epic_status WitnessLaunch<W>::run(epic_ctx* c, const int32_t* seqs, int B, int n, uint8_t* bytes, int bytes_per_seq,
                                  int32_t* gap_len, int max_gaps, int32_t* status, void* wws, void* ws,
                                  hipStream_t stream) {
  const WsArgs wa = ws_args(c, ws);
  const WitArgs wt = wit_args(c, wws);
  hipLaunchKernelGGL((witness_walk_kernel<W, kThreads>), dim3(B), dim3(kThreads), 0, stream, c->tab, seqs, B, n, wa,
                     wt, status);
  hipLaunchKernelGGL((witness_trace_kernel<W>), dim3(B), dim3(64), 0, stream, c->tab, wa, wt, status, B);
  hipLaunchKernelGGL((witness_realize_kernel<256>), dim3(B), dim3(256), 0, stream, c->tab, seqs, B, n, wt, status,
                     bytes, bytes_per_seq, gap_len, max_gaps);
  return hipGetLastError() == hipSuccess ? EPIC_OK : EPIC_ERR_HIP;
}

template struct WitnessLaunch<EPIC_KERNEL_UNIT>;
template struct ValidatePlainLaunch<EPIC_KERNEL_UNIT>;
template struct ValidateLaunch<EPIC_KERNEL_UNIT>;
template struct FallbackLaunch<EPIC_KERNEL_UNIT>;
template struct SelectLaunch<EPIC_KERNEL_UNIT>;
#else

// Device scratch of epic_validate_batch_noalloc, for callers that cannot
// allocate: a file-scope array, one copy per GPU, held until the process
// ends.  Host code never passes `scratch` itself to a kernel (on the host it
// names a stand-in, not device memory): each device's address comes from
// hipGetSymbolAddress, taken once per device with that device current.
constexpr size_t kStaticScratchBytes = (size_t)256 << 20;
static __device__ __align__(256) char scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
constexpr int kMaxDevices = 64;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address (set-up, once per device); nullptr
// if the lookup fails.
void* device_scratch(int device) {
  if (device < 0 || device >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[device]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) {
      (void)hipGetLastError();
      return nullptr;
    }
    g_scratch_ptr[device] = p;
  }
  return g_scratch_ptr[device];
}
}  // namespace

template <template <int> class Launcher, class... Args>
epic_status dispatch_w(int W, Args... args) {
  switch (W) {
    case 1: return Launcher<1>::run(args...);
    case 2: return Launcher<2>::run(args...);
    case 4: return Launcher<4>::run(args...);
    case 8: return Launcher<8>::run(args...);
    case 16: return Launcher<16>::run(args...);
    default: return EPIC_ERR_UNSUPPORTED;
  }
}

// LDS streaming microbenchmark (epic_diag_lds_stream): 64 KiB of LDS read
// as 16-byte vectors at consecutive addresses per wavefront.  The stride and
// the index mask are kernel arguments, so no two reads of the loop are known
// to the compiler to hit the same address (none is merged away).
__global__ void __launch_bounds__(1024) lds_stream_kernel(int iters, int stride, int mask,
                                                          uint32_t* __restrict__ sink) {
  __shared__ uint4 buf[4096];
  const int t = (int)threadIdx.x, nt = (int)blockDim.x;
  for (int i = t; i < 4096; i += nt) buf[i] = make_uint4((uint32_t)i, 3u * i, 5u * i, 7u * i);
  __syncthreads();
  const long long c0 = (long long)clock64(), w0 = (long long)wall_clock64();
  uint32_t a0 = 0, a1 = 0, a2 = 0, a3 = 0;
  int idx = t;
#pragma unroll 8
  for (int k = 0; k < iters; ++k) {
    const uint4 v = buf[idx & mask];
    a0 += v.x;
    a1 += v.y;
    a2 += v.z;
    a3 += v.w;
    idx += stride;
  }
  const long long c1 = (long long)clock64(), w1 = (long long)wall_clock64();
  if ((a0 ^ a1 ^ a2 ^ a3) == 0x9E3779B9u) sink[0] = 1u;  // keeps the reads
  if (blockIdx.x == 0 && t == 0) {
    const unsigned long long dc = (unsigned long long)(c1 - c0), dw = (unsigned long long)(w1 - w0);
    sink[2] = (uint32_t)dc;
    sink[3] = (uint32_t)(dc >> 32);
    sink[4] = (uint32_t)dw;
    sink[5] = (uint32_t)(dw >> 32);
  }
}

extern "C" {

static epic_status read_counters(epic_ctx* c, hipStream_t stream, int64_t* sets) {
  if (hipStreamSynchronize(stream) != hipSuccess) return EPIC_ERR_HIP;
  if (hipMemcpy(sets, (char*)c->d_err + kWorkOff, kKernelKinds * 8 * sizeof(int64_t), hipMemcpyDeviceToHost) !=
      hipSuccess)
    return EPIC_ERR_HIP;
  if (hipMemset((char*)c->d_err + kWorkOff, 0, kKernelKinds * 8 * sizeof(int64_t)) != hipSuccess) return EPIC_ERR_HIP;
  return EPIC_OK;
}

epic_status epic_ctx_work_counters(epic_ctx* c, hipStream_t stream, int64_t* out) {
  if (!c || !out) return EPIC_ERR_NULL;
  int64_t sets[kKernelKinds * 8];
  epic_status s = read_counters(c, stream, sets);
  if (s != EPIC_OK) return s;
  for (int i = 0; i < kWorkCounters; ++i) {
    out[i] = 0;
    for (int k = 0; k < kKernelKinds; ++k) out[i] += sets[k * 8 + i];
  }
  return EPIC_OK;
}

epic_status epic_ctx_set_timing(epic_ctx* c, int32_t enable) {
  if (!c) return EPIC_ERR_NULL;
  c->timing = enable != 0;
  return EPIC_OK;
}

epic_status epic_ctx_set_witness_lds(epic_ctx* c, int32_t max_proofs, int32_t max_vis_words) {
  if (!c) return EPIC_ERR_NULL;
  if (max_proofs < 0 || max_proofs > kWitLdsSlots / 2 || max_vis_words < 0 || max_vis_words > kWitVisLds)
    return EPIC_ERR_ARG;
  c->wit_lds_proofs = max_proofs;
  c->wit_lds_vis = max_vis_words;
  return EPIC_OK;
}

epic_status epic_ctx_kernel_stats(epic_ctx* c, hipStream_t stream, double* ms, int64_t* launches, int64_t* work) {
  if (!c || !ms || !launches || !work) return EPIC_ERR_NULL;
  int64_t sets[kKernelKinds * 8];
  epic_status s = read_counters(c, stream, sets);
  if (s != EPIC_OK) return s;
  for (auto& p : c->pending) {
    float t = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&t, p.a, p.b) == hipSuccess) {
      c->kernel_ms[p.kid] += t;
      c->kernel_launches[p.kid] += 1;
    }
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  c->pending.clear();
  for (int k = 0; k < kKernelKinds; ++k) {
    ms[k] = c->kernel_ms[k];
    launches[k] = c->kernel_launches[k];
    c->kernel_ms[k] = 0;
    c->kernel_launches[k] = 0;
    for (int i = 0; i < kWorkCounters; ++i) work[k * kWorkCounters + i] = sets[k * 8 + i];
  }
  return EPIC_OK;
}

epic_status epic_diag_lds_stream(int32_t blocks, int32_t threads, int32_t iters, uint32_t* d_sink,
                                 hipStream_t stream) {
  if (!d_sink) return EPIC_ERR_NULL;
  if (blocks < 1 || blocks > (1 << 20) || threads < 64 || threads > 1024 || threads % 64 != 0 || iters < 1)
    return EPIC_ERR_ARG;
  hipLaunchKernelGGL(lds_stream_kernel, dim3(blocks), dim3(threads), 0, stream, (int)iters, (int)threads, 4095, d_sink);
  return hipGetLastError() == hipSuccess ? EPIC_OK : EPIC_ERR_HIP;
}

epic_status epic_diag_clock_rates(int32_t* shader_khz, int32_t* wall_khz) {
  if (!shader_khz || !wall_khz) return EPIC_ERR_NULL;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return EPIC_ERR_HIP;
  if (hipDeviceGetAttribute(shader_khz, hipDeviceAttributeClockRate, dev) != hipSuccess) return EPIC_ERR_HIP;
  if (hipDeviceGetAttribute(wall_khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess) return EPIC_ERR_HIP;
  return EPIC_OK;
}

const char* epic_status_string(epic_status s) {
  switch (s) {
    case EPIC_OK: return "ok";
    case EPIC_ERR_NULL: return "null pointer";
    case EPIC_ERR_ARG: return "argument out of range";
    case EPIC_ERR_CAPACITY: return "capacity exceeded";
    case EPIC_ERR_LEXER: return "malformed lexer DFA";
    case EPIC_ERR_GRAMMAR: return "malformed grammar";
    case EPIC_ERR_VOCAB: return "malformed vocabulary";
    case EPIC_ERR_HIP: return "HIP runtime error";
    case EPIC_ERR_STATE: return "memo not built";
    case EPIC_ERR_UNSUPPORTED: return "unsupported size";
  }
  return "unknown status";
}

epic_status epic_ctx_create(const epic_lexer_desc* lexer, const epic_grammar_desc* grammar,
                            const epic_vocab_desc* vocab, int32_t max_batch, int32_t max_seq_len, int32_t max_cands,
                            epic_ctx** out) {
  if (!lexer || !grammar || !vocab || !out || !lexer->trans || !lexer->accept || !grammar->lhs ||
      !grammar->rhs_offsets || !vocab->bytes || !vocab->offsets)
    return EPIC_ERR_NULL;
  if (grammar->num_productions > 0 && grammar->rhs_offsets[grammar->num_productions] > 0 && !grammar->rhs)
    return EPIC_ERR_NULL;
  *out = nullptr;
  if (max_batch < 1 || max_seq_len < 1 || max_cands < 1) return EPIC_ERR_ARG;
  if (max_seq_len > kMaxSeq) return EPIC_ERR_UNSUPPORTED;
  epic_ctx* c = new epic_ctx();
  std::string why;
  int r = build_tables(lexer->num_states, lexer->trans, lexer->accept, grammar->num_terminals,
                       grammar->num_nonterminals, grammar->start, grammar->num_productions, grammar->lhs,
                       grammar->rhs_offsets, grammar->rhs, vocab->vocab_size, vocab->bytes, vocab->offsets, c->H, why);
  if (r != 0) {
    delete c;
    return (epic_status)r;
  }
  if (hipGetDevice(&c->device) != hipSuccess) c->device = 0;
  if (hipDeviceGetAttribute(&c->num_cus, hipDeviceAttributeMultiprocessorCount, c->device) != hipSuccess ||
      c->num_cus < 1)
    c->num_cus = 256;
  c->max_batch = max_batch;
  c->max_seq = max_seq_len;
  c->max_cands = max_cands;
  const HostTables& H = c->H;
  // graph nodes: start, final, one per fixed byte, K per masked run
  c->maxn = 8 * max_seq_len + H.K * (max_seq_len / 2 + 2) + 4;
  c->maxe = std::min(std::max(16384, 512 * max_seq_len), 131072);
  c->nslot = std::min(std::max(max_cands, max_batch), 1024);
  c->off_cnt = align256((size_t)c->maxn * 4);
  c->off_org = c->off_cnt + align256((size_t)c->maxn * 4);
  c->off_sn = c->off_org + align256((size_t)c->maxe * 4);
  c->off_st = c->off_sn + align256((size_t)c->maxe * 8);
  c->off_bits = c->off_st + align256((size_t)c->maxe * 8);
  c->off_cov = c->off_bits + align256((size_t)c->maxe * H.W * 4);
  c->slot_bytes = c->off_cov + align256((size_t)c->maxn * H.CW * 4);
  c->base_slots = std::min(max_batch, 1024);
  c->snap_bytes = align256(kSnapHeader + (size_t)(max_seq_len / 2 + 1) * sizeof(Snapshot));
  c->off_snap = c->slot_bytes * (size_t)(c->nslot + 2 * c->base_slots);
  c->off_bseq = c->off_snap + c->snap_bytes * 2 * c->base_slots;
  c->off_spec = c->off_bseq + align256((size_t)2 * c->base_slots * max_seq_len * 4);
  c->ws_bytes = c->off_spec + align256((size_t)spec_words(c->max_batch) * 4);  // + speculated checks
  // witness workspace, per sequence: edge record, on-path marks (one bit per
  // chart item), search stack, witness terminals, byte-search records and
  // visited set, stored proofs and their index
  c->wit_ecap = 4 * c->maxn + 4096;
  c->wit_rec = 0;
  c->wit_mark = align256((size_t)4 * (kRecHeader + 4 * (size_t)c->maxn + 4 * (size_t)c->wit_ecap));
  c->wit_stack = c->wit_mark + align256((size_t)c->maxe * H.W * 4);
  c->wit_w = c->wit_stack + align256((size_t)kWitFrames * sizeof(WitFrame));
  c->wit_recs = c->wit_w + align256((size_t)(kWitTerminals + 1) * 4);
  c->wit_vis = c->wit_recs + align256((size_t)kWitRecords * sizeof(WitRec));
  c->wit_proof = c->wit_vis + align256((size_t)kWitVisWords * 4);
  c->wit_pindex = c->wit_proof + align256((size_t)kWitProofs * sizeof(WitProof));
  c->wit_sys = c->wit_pindex + align256((size_t)kWitProofSlots * 4);
  c->wit_stride = c->wit_sys + align256((size_t)kWitSystems * 8 + (size_t)2 * kWitSystems * 4 + 256 * 4 +
                                        (size_t)kWitSystems * std::max(H.K, 1) * H.NI * 2);
  epic_status s = upload(c);
  if (s != EPIC_OK) {
    epic_ctx_destroy(c);
    return s;
  }
  c->scratch = device_scratch(c->device);  // with the context's device current
  *out = c;
  return EPIC_OK;
}

void epic_ctx_destroy(epic_ctx* c) {
  if (!c) return;
  for (auto& p : c->pending) {
    (void)hipEventDestroy(p.a);
    (void)hipEventDestroy(p.b);
  }
  if (c->d_tables) (void)hipFree(c->d_tables);
  if (c->d_memo) (void)hipFree(c->d_memo);
  if (c->d_err) (void)hipFree(c->d_err);
  delete c;
}

size_t epic_workspace_bytes(const epic_ctx* c) { return c ? c->ws_bytes : 0; }

int32_t epic_gap_classes(const epic_ctx* c) { return c ? c->H.K : -1; }

int32_t epic_item_words(const epic_ctx* c) { return c ? c->H.W : -1; }

epic_status epic_lexmemo_build(epic_ctx* c, hipStream_t stream) {
  if (!c) return EPIC_ERR_NULL;
  const size_t total = (size_t)c->H.V * c->H.Q;
  const unsigned grid = (unsigned)((total + kMemoThreads - 1) / kMemoThreads);
  {
    KernelTimer kt(c, kKLexmemo, stream);
    hipLaunchKernelGGL(lexmemo_kernel, dim3(grid), dim3(kMemoThreads), 0, stream, c->tab, c->d_memo);
  }
  if (hipGetLastError() != hipSuccess) return EPIC_ERR_HIP;
  c->memo_built = true;
  return EPIC_OK;
}

epic_status epic_memo_export(const epic_ctx* c, void* host_dst, size_t bytes) {
  if (!c || !host_dst) return EPIC_ERR_NULL;
  if (!c->memo_built) return EPIC_ERR_STATE;
  const size_t need = (size_t)c->H.V * c->H.Q * 16;
  if (bytes < need) return EPIC_ERR_CAPACITY;
  if (hipDeviceSynchronize() != hipSuccess) return EPIC_ERR_HIP;
  if (hipMemcpy(host_dst, c->d_memo, need, hipMemcpyDeviceToHost) != hipSuccess) return EPIC_ERR_HIP;
  return EPIC_OK;
}

static epic_status check_batch(const epic_ctx* c, const int32_t* seqs, int B, int n, const int32_t* cs,
                               const int32_t* cp, const int32_t* ct, int C, const void* out, const void* ws,
                               size_t ws_bytes) {
  if (!c) return EPIC_ERR_NULL;
  if (B < 0 || n < 0 || C < 0) return EPIC_ERR_ARG;
  if (B > c->max_batch || n > c->max_seq || C > c->max_cands) return EPIC_ERR_CAPACITY;
  if (C == 0) return EPIC_OK;
  if (!seqs || !cs || !cp || !ct || !out || !ws) return EPIC_ERR_NULL;
  if (((uintptr_t)ws & 255) != 0) return EPIC_ERR_ARG;
  if (ws_bytes < c->ws_bytes) return EPIC_ERR_CAPACITY;
  if (!c->memo_built) return EPIC_ERR_STATE;
  return EPIC_OK;
}

epic_status epic_validate_batch(epic_ctx* c, const int32_t* d_seqs, int32_t B, int32_t n, const int32_t* d_cand_seq,
                                const int32_t* d_cand_pos, const int32_t* d_cand_tok, int32_t C, uint8_t* d_verdict,
                                void* d_workspace, size_t workspace_bytes, hipStream_t stream) {
  epic_status s =
      check_batch(c, d_seqs, B, n, d_cand_seq, d_cand_pos, d_cand_tok, C, d_verdict, d_workspace, workspace_bytes);
  if (s != EPIC_OK || C == 0) return s;
  return dispatch_w<ValidateLaunch>(c->H.W, c, d_seqs, (int)B, (int)n, d_cand_seq, d_cand_pos, d_cand_tok, (int)C,
                                    d_verdict, d_workspace, stream);
}

epic_status epic_validate_batch_noalloc(epic_ctx* c, const int32_t* d_seqs, int32_t B, int32_t n,
                                        const int32_t* d_cand_seq, const int32_t* d_cand_pos,
                                        const int32_t* d_cand_tok, int32_t C, uint8_t* d_verdict,
                                        hipStream_t stream) {
  if (!c) return EPIC_ERR_NULL;
  if (B < 0 || n < 0 || C < 0) return EPIC_ERR_ARG;
  if (B > c->max_batch || n > c->max_seq || C > c->max_cands) return EPIC_ERR_CAPACITY;
  if (C == 0) return EPIC_OK;
  if (!d_seqs || !d_cand_seq || !d_cand_pos || !d_cand_tok || !d_verdict) return EPIC_ERR_NULL;
  if (!c->memo_built) return EPIC_ERR_STATE;
  if (!c->scratch) return EPIC_ERR_HIP;
  const size_t nslot = kStaticScratchBytes / c->slot_bytes;  // walks resident at once
  if (nslot < 1) return EPIC_ERR_CAPACITY;  // one walk's chart does not fit
  return dispatch_w<ValidatePlainLaunch>(c->H.W, c, d_seqs, (int)B, (int)n, d_cand_seq, d_cand_pos, d_cand_tok, (int)C,
                                         d_verdict, c->scratch, (int)std::min<size_t>(nslot, 1024), stream);
}

epic_status epic_select_compatible(epic_ctx* c, const int32_t* d_seqs, int32_t B, int32_t n,
                                   const int32_t* d_cand_seq, const int32_t* d_cand_pos, const int32_t* d_cand_tok,
                                   const float* d_conf, const uint8_t* d_verdict, int32_t C, uint8_t* d_selected,
                                   int64_t* d_counts, void* d_workspace, size_t workspace_bytes, hipStream_t stream) {
  epic_status s =
      check_batch(c, d_seqs, B, n, d_cand_seq, d_cand_pos, d_cand_tok, C, d_selected, d_workspace, workspace_bytes);
  if (s != EPIC_OK || C == 0 || B == 0) return s;
  if (!d_conf || !d_verdict) return EPIC_ERR_NULL;
  if (B > c->nslot) return EPIC_ERR_CAPACITY;
  return dispatch_w<SelectLaunch>(c->H.W, c, d_seqs, (int)B, (int)n, d_cand_seq, d_cand_pos, d_cand_tok, d_conf,
                                  d_verdict, (int)C, d_selected, d_counts, d_workspace, stream);
}

epic_status epic_commit_fallback(epic_ctx* c, const int32_t* d_seqs, int32_t B, int32_t n,
                                 const int32_t* d_cand_seq, const int32_t* d_cand_pos, const int32_t* d_cand_tok,
                                 const float* d_conf, const uint8_t* d_verdict, const uint8_t* d_selected,
                                 const int32_t* d_num_commit, int32_t C, uint8_t* d_accepted, void* d_workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  epic_status s =
      check_batch(c, d_seqs, B, n, d_cand_seq, d_cand_pos, d_cand_tok, C, d_accepted, d_workspace, workspace_bytes);
  if (s != EPIC_OK || C == 0 || B == 0) return s;
  if (!d_conf || !d_verdict || !d_selected || !d_num_commit) return EPIC_ERR_NULL;
  return dispatch_w<FallbackLaunch>(c->H.W, c, d_seqs, (int)B, (int)n, d_cand_seq, d_cand_pos, d_cand_tok, d_conf,
                                    d_verdict, d_selected, d_num_commit, (int)C, d_accepted, d_workspace, stream);
}

size_t epic_witness_workspace_bytes(const epic_ctx* c, int32_t B) {
  return c && B > 0 ? c->wit_stride * (size_t)B : 0;
}

epic_status epic_witness(epic_ctx* c, const int32_t* d_seqs, int32_t B, int32_t n, uint8_t* d_bytes,
                         int32_t bytes_per_seq, int32_t* d_gap_len, int32_t max_gaps, int32_t* d_status,
                         void* d_witness_ws, size_t witness_ws_bytes, void* d_workspace, size_t workspace_bytes,
                         hipStream_t stream) {
  if (!c) return EPIC_ERR_NULL;
  if (B < 0 || n < 1 || bytes_per_seq < 0 || max_gaps < 1) return EPIC_ERR_ARG;
  if (B > c->max_batch || B > c->nslot || n > c->max_seq) return EPIC_ERR_CAPACITY;
  if (B == 0) return EPIC_OK;
  if (!d_seqs || !d_bytes || !d_gap_len || !d_status || !d_witness_ws || !d_workspace) return EPIC_ERR_NULL;
  if (((uintptr_t)d_workspace & 255) != 0 || ((uintptr_t)d_witness_ws & 255) != 0) return EPIC_ERR_ARG;
  if (workspace_bytes < c->ws_bytes || witness_ws_bytes < c->wit_stride * (size_t)B) return EPIC_ERR_CAPACITY;
  if (!c->memo_built) return EPIC_ERR_STATE;
  return dispatch_w<WitnessLaunch>(c->H.W, c, d_seqs, (int)B, (int)n, d_bytes, (int)bytes_per_seq, d_gap_len,
                                   (int)max_gaps, d_status, d_witness_ws, d_workspace, stream);
}

epic_status epic_ctx_device_error(epic_ctx* c, hipStream_t stream, uint32_t* flags) {
  if (!c || !flags) return EPIC_ERR_NULL;
  if (hipStreamSynchronize(stream) != hipSuccess) return EPIC_ERR_HIP;
  uint32_t v = 0;
  if (hipMemcpy(&v, c->d_err, 4, hipMemcpyDeviceToHost) != hipSuccess) return EPIC_ERR_HIP;
  if (hipMemset(c->d_err, 0, 4) != hipSuccess) return EPIC_ERR_HIP;
  *flags = v;
  return EPIC_OK;
}

}  // extern "C"
#endif  // EPIC_KERNEL_UNIT
