// Host driver of the encrypted affine prefix scan of HEScan (Sec. "Parallel
// Prefix Scans", paragraph "Affine Prefix Composition", Eq.
// "compact_affine_compose"; Brent-Kung network of Appendix "Prefix-Network
// Selection"; Sec. "Resident Block Schedule", Eq. "resident-block-schedule").
//
// A token map is the ciphertext pair (a, s) for F(z) = a z + s; R after L
// composes to (a_R a_L, a_R s_L + s_R).  One composition is two products at
// the lower level l of its operands, each relinearised and divided by
// P q_{l-1} in one step (ModDown merged with the rescale):
//     a' = a_R a_L / (P q_{l-1}),   s' = a_R s_L / (P q_{l-1}) + s_R   (level l - 1)
// where s_R enters through its first l - 1 limbs.  Ciphertexts are
// [level][2][N] limb-major, so dropping to a lower level is taking a prefix of
// the buffer: no copies are made for it.
//
// Every stage of the network is one batch: its nodes are independent (no
// node reads a position another node of the stage writes), so the nodes of a
// stage, over all chunks, are grouped by level and run as batched products
// (op_prod_rescale_many: one key switch per 32 products, sharing the
// relinearisation key, with the tensor formed inside and s_R added in the
// final combine).  A node's state product is issued before its decay product,
// so the node may write in place over the operands it reads.
#include <algorithm>
#include <map>
#include <vector>

#include "fesc_internal.hpp"
#include "ops.hpp"

namespace fesc {

namespace {

#define HIPCK_RET(expr)                                \
  do {                                                 \
    hipError_t e_ = (expr);                            \
    if (e_ != hipSuccess) return hip_check(e_, #expr); \
  } while (0)

struct Node {
  uint32_t dst, src;  // 0-based positions; dst takes src o dst
};
using Stages = std::vector<std::vector<Node>>;

// Brent-Kung network over L positions (padded to L' = 2^ceil(log2 L); nodes
// whose destination lies past L are left out: no node reads a position above
// its destination, so valid prefixes do not depend on them).  Up-sweep stage
// s: each 2^s-aligned position takes the one 2^(s-1) to its left; down-sweep
// stage s: each multiple k of 2^s passes its prefix to k + 2^(s-1).
Stages bk_network(uint32_t L) {
  Stages st;
  if (L < 2) return st;
  uint32_t m = 0;
  while ((1u << m) < L) ++m;
  const uint32_t Lp = 1u << m;
  for (uint32_t s = 1; s <= m; ++s) {
    std::vector<Node> v;
    for (uint32_t k = 1u << s; k <= Lp; k += 1u << s)
      if (k <= L) v.push_back(Node{k - 1, k - 1 - (1u << (s - 1))});
    st.push_back(v);
  }
  for (uint32_t s = m - 1; s >= 1; --s) {
    std::vector<Node> v;
    for (uint32_t k = 1u << s; k <= Lp; k += 1u << s) {
      const uint32_t j = k + (1u << (s - 1));
      if (j <= L) v.push_back(Node{j - 1, k - 1});
    }
    st.push_back(v);
  }
  return st;
}

// Only the nodes the last position depends on (a block summary).
Stages prune_to_last(const Stages& st, uint32_t L) {
  std::vector<char> need(L, 0);
  need[L - 1] = 1;
  Stages out(st.size());
  for (size_t i = st.size(); i-- > 0;)
    for (const Node& nd : st[i])
      if (need[nd.dst]) {
        out[i].push_back(nd);
        need[nd.src] = 1;
      }
  return out;
}

// Which decay products are needed.  A node (dst <- src o dst) always forms
// its state product a_dst s_src (every state is an output or feeds one); its
// decay product a_dst a_src only if a later product reads the new a_dst.
// need[p]: the final decay of position p is wanted by the caller.  Walking
// the nodes backwards: the decay product of a node is live iff its dst's
// decay is needed afterwards; a node's products read the old a_dst (always)
// and a_src (if the decay product is live).  Returns per stage, per node.
std::vector<std::vector<char>> live_decay(const Stages& st, std::vector<char> need) {
  std::vector<std::vector<char>> live(st.size());
  for (size_t i = 0; i < st.size(); ++i) live[i].assign(st[i].size(), 0);
  for (size_t i = st.size(); i-- > 0;)
    for (size_t j = st[i].size(); j-- > 0;) {
      const Node& nd = st[i][j];
      live[i][j] = need[nd.dst];
      if (live[i][j]) need[nd.src] = 1;
      need[nd.dst] = 1;
    }
  return live;
}

// Decay needs at the start of a network (before any node), given the final
// needs: which input decays the network reads.
std::vector<char> decay_needed_at_start(const Stages& st, std::vector<char> need) {
  for (size_t i = st.size(); i-- > 0;)
    for (size_t j = st[i].size(); j-- > 0;) {
      const Node& nd = st[i][j];
      if (need[nd.dst]) need[nd.src] = 1;
      need[nd.dst] = 1;
    }
  return need;
}

// One chunk's positions: the buffers holding their current values and the
// buffers a composition writes to.
struct Seq {
  std::vector<const uint64_t*> cur_a, cur_s;
  std::vector<uint64_t*> home_a, home_s;
};

// The products a driver issues, recorded instead of launched (host-side
// verification of the schedule with placeholder buffer addresses): per
// product (group, x, y, add or 0, out) for out = x y (+ add); a copy is
// (group, src, 0, 0, dst).  Products of one group are one batched call, whose
// operands are all read before any output is written.
struct Program {
  std::vector<uint64_t> words;
  uint64_t group = 0;
  void product(const uint64_t* x, const uint64_t* y, const uint64_t* add, const uint64_t* out) {
    for (uint64_t w : {group, (uint64_t)(uintptr_t)x, (uint64_t)(uintptr_t)y,
                       (uint64_t)(uintptr_t)add, (uint64_t)(uintptr_t)out})
      words.push_back(w);
  }
};

// Runs the stages over all chunks; lvl[] (shared by the chunks, which have
// the same structure) tracks each position's level.  need_final[p]: the
// caller wants position p's final decay (dead decay products are skipped).
// dry: levels only.  Each node's state product is issued before its decay
// product: the state product reads the old a_dst and writes only s_dst,
// which the decay product does not read, so the two may fall in different
// product groups.
int run_stages(Context* c, const Stages& st, std::vector<Seq>& seqs, std::vector<uint32_t>& lvl,
               const std::vector<char>& need_final, bool dry, hipStream_t s,
               uint64_t* nprod = nullptr, Program* prog = nullptr) {
  const std::vector<std::vector<char>> live = live_decay(st, need_final);
  if (nprod)
    for (size_t i = 0; i < st.size(); ++i)
      for (size_t j = 0; j < st[i].size(); ++j) *nprod += 1 + live[i][j];
  for (size_t si = 0; si < st.size(); ++si) {
    std::map<uint32_t, std::vector<uint32_t>> by_level;  // node indices of the stage
    for (uint32_t j = 0; j < st[si].size(); ++j) {
      const Node& nd = st[si][j];
      by_level[std::min(lvl[nd.dst], lvl[nd.src])].push_back(j);
    }
    for (const auto& kv : by_level) {
      const uint32_t l = kv.first;
      if (l < 2) return fail(FESC_ERR_LEVEL, "affine scan needs more levels than the input has");
      if (!dry) {
        std::vector<const uint64_t*> xs, ys, adds;
        std::vector<uint64_t*> outs;
        for (Seq& q : seqs)
          for (uint32_t j : kv.second) {
            const Node& nd = st[si][j];
            xs.push_back(q.cur_a[nd.dst]);
            ys.push_back(q.cur_s[nd.src]);
            outs.push_back(q.home_s[nd.dst]);
            adds.push_back(q.cur_s[nd.dst]);
            if (!live[si][j]) continue;
            xs.push_back(q.cur_a[nd.dst]);
            ys.push_back(q.cur_a[nd.src]);
            outs.push_back(q.home_a[nd.dst]);
            adds.push_back(nullptr);
          }
        if (prog) {
          for (size_t i = 0; i < xs.size(); ++i) prog->product(xs[i], ys[i], adds[i], outs[i]);
          ++prog->group;
        } else {
          int err = op_prod_rescale_many(c, (uint32_t)xs.size(), xs.data(), ys.data(),
                                         outs.data(), adds.data(), l, l - 1, s);
          if (err) return err;
        }
      }
      for (uint32_t j : kv.second) {
        const Node& nd = st[si][j];
        for (Seq& q : seqs) {
          q.cur_a[nd.dst] = live[si][j] ? q.home_a[nd.dst] : nullptr;  // dead: never read
          q.cur_s[nd.dst] = q.home_s[nd.dst];
        }
        lvl[nd.dst] = l - 1;
      }
    }
  }
  return FESC_OK;
}


uint32_t min_level(const std::vector<uint32_t>& lvl) {
  return *std::min_element(lvl.begin(), lvl.end());
}

}  // namespace

size_t affine_scan_network(uint32_t L, bool states_only, uint32_t* nodes, size_t cap) {
  const Stages net = bk_network(L);
  const std::vector<std::vector<char>> live =
      live_decay(net, std::vector<char>(L, states_only ? 0 : 1));
  size_t k = 0;
  for (size_t i = 0; i < net.size(); ++i)
    for (size_t j = 0; j < net[i].size(); ++j, ++k)
      if (nodes && k < cap) {
        uint32_t* o = nodes + 4 * k;
        o[0] = (uint32_t)i;
        o[1] = net[i][j].dst;
        o[2] = net[i][j].src;
        o[3] = (uint32_t)live[i][j];
      }
  return k;
}

int op_affine_scan_level(Context* c, uint32_t L, uint32_t level, bool states_only,
                         uint32_t* out_level, uint64_t* products) {
  const Stages net = bk_network(L);
  std::vector<uint32_t> lvl(L, level);
  std::vector<Seq> none;
  *products = 0;
  int err = run_stages(c, net, none, lvl, std::vector<char>(L, states_only ? 0 : 1), true,
                       nullptr, products);
  if (err) return err;
  *out_level = min_level(lvl);
  return FESC_OK;
}

// The in-place scan of `chunks` sequences; prog: record instead of launch.
static int scan_in_place(Context* c, uint64_t* const* a, uint64_t* const* s, uint32_t L,
                         uint32_t chunks, uint32_t level, bool states_only, uint32_t* out_level,
                         hipStream_t st, Program* prog) {
  const Stages net = bk_network(L);
  const std::vector<char> need(L, states_only ? 0 : 1);
  std::vector<uint32_t> lvl(L, level);
  std::vector<Seq> none;
  int err;
  if ((err = run_stages(c, net, none, lvl, need, true, st))) return err;
  std::vector<Seq> seqs(chunks);
  for (uint32_t ch = 0; ch < chunks; ++ch) {
    Seq& q = seqs[ch];
    for (uint32_t k = 0; k < L; ++k) {
      q.cur_a.push_back(a[(size_t)ch * L + k]);
      q.cur_s.push_back(s[(size_t)ch * L + k]);
      q.home_a.push_back(a[(size_t)ch * L + k]);
      q.home_s.push_back(s[(size_t)ch * L + k]);
    }
  }
  lvl.assign(L, level);
  if ((err = run_stages(c, net, seqs, lvl, need, false, st, nullptr, prog))) return err;
  *out_level = min_level(lvl);
  return FESC_OK;
}

int op_affine_scan(Context* c, uint64_t* const* a, uint64_t* const* s, uint32_t L,
                   uint32_t chunks, uint32_t level, bool states_only, uint32_t* out_level,
                   hipStream_t st) {
  return scan_in_place(c, a, s, L, chunks, level, states_only, out_level, st, nullptr);
}


size_t affine_scan_resident_words(const Context* c, uint32_t L, uint32_t chunks, uint32_t block,
                                  uint32_t level) {
  const size_t K = (L + block - 1) / block;
  return (size_t)chunks * (2 * block + 2 * (K - 1)) * 2 * level * c->n;
}

// Two passes over blocks of `block` tokens: pass 1 builds the summary (last
// local prefix) of every block but the last, an exclusive scan over the
// summaries (the same network) gives the carries G_j, pass 2 replays each
// block and writes the states of its corrected prefixes P_{j,t} o G_j:
//     h = a_P G_s + s_P  (j >= 1),   h = s_P  (j = 0).
// The workspace holds, per chunk, one block of tuples and the summaries:
// [chunk][2 block + 2 (K - 1)][level][2][N].
static int resident(Context* c, const uint64_t* const* a, const uint64_t* const* s, uint32_t L,
                    uint32_t chunks, uint32_t block, uint64_t* const* h, uint32_t level,
                    uint32_t out_level, uint64_t* ws, bool dry, uint32_t* min_out,
                    hipStream_t st, uint64_t* nprod = nullptr, Program* prog = nullptr) {
  const uint32_t K = (L + block - 1) / block;
  // recording: one placeholder word per workspace slot
  const size_t W = prog ? 1 : (size_t)2 * level * c->n;
  const size_t per_chunk = (size_t)(2 * block + 2 * (K - 1)) * W;
  auto blk_a = [&](uint32_t ch, uint32_t t) { return ws + ch * per_chunk + (size_t)t * W; };
  auto blk_s = [&](uint32_t ch, uint32_t t) {
    return ws + ch * per_chunk + (size_t)(block + t) * W;
  };
  auto sum_a = [&](uint32_t ch, uint32_t j) {
    return ws + ch * per_chunk + (size_t)(2 * block + j) * W;
  };
  auto sum_s = [&](uint32_t ch, uint32_t j) {
    return ws + ch * per_chunk + (size_t)(2 * block + (K - 1) + j) * W;
  };
  auto in_seq = [&](uint32_t ch, uint32_t j, uint32_t Bj, bool summary) {
    Seq q;
    for (uint32_t t = 0; t < Bj; ++t) {
      const size_t idx = (size_t)ch * L + (size_t)j * block + t;
      q.cur_a.push_back(dry ? nullptr : a[idx]);
      q.cur_s.push_back(dry ? nullptr : s[idx]);
      const bool last = summary && t == Bj - 1;
      q.home_a.push_back(dry ? nullptr : last ? sum_a(ch, j) : blk_a(ch, t));
      q.home_s.push_back(dry ? nullptr : last ? sum_s(ch, j) : blk_s(ch, t));
    }
    return q;
  };
  const uint32_t nseq = dry ? 1 : chunks;
  int err;
  // decays needed: the carries are used through their states only; the
  // carry network then says which summary decays it reads
  const Stages carry_net = K > 1 ? bk_network(K - 1) : Stages{};
  const std::vector<char> carry_need(K > 1 ? K - 1 : 0, 0);
  const std::vector<char> sum_need = decay_needed_at_start(carry_net, carry_need);
  // pass 1: summaries of blocks 0 .. K-2
  const Stages summary_net = prune_to_last(bk_network(block), block);
  std::vector<Seq> carry(nseq);
  std::vector<uint32_t> lvl_sum;
  for (uint32_t j = 0; j + 1 < K; ++j) {
    std::vector<Seq> seqs;
    for (uint32_t ch = 0; ch < nseq; ++ch) seqs.push_back(in_seq(ch, j, block, true));
    std::vector<uint32_t> lvl(block, level);
    std::vector<char> need(block, 0);
    need[block - 1] = sum_need[j];
    if ((err = run_stages(c, summary_net, seqs, lvl, need, dry, st, nprod, prog))) return err;
    lvl_sum.push_back(lvl[block - 1]);
    for (uint32_t ch = 0; ch < nseq; ++ch) {
      carry[ch].cur_a.push_back(seqs[ch].cur_a[block - 1]);
      carry[ch].cur_s.push_back(seqs[ch].cur_s[block - 1]);
      carry[ch].home_a.push_back(dry ? nullptr : sum_a(ch, j));
      carry[ch].home_s.push_back(dry ? nullptr : sum_s(ch, j));
    }
  }
  // exclusive scan over the summaries: G_j = carry position j - 1
  if (K > 1 &&
      (err = run_stages(c, carry_net, carry, lvl_sum, carry_need, dry, st, nprod, prog)))
    return err;
  // pass 2: replay and carry injection
  uint32_t lo = level;
  for (uint32_t j = 0; j < K; ++j) {
    const uint32_t Bj = std::min(block, L - j * block);
    std::vector<Seq> seqs;
    for (uint32_t ch = 0; ch < nseq; ++ch) seqs.push_back(in_seq(ch, j, Bj, false));
    std::vector<uint32_t> lvl(Bj, level);
    // block 0 gives states; later blocks' decays enter the carry injection
    const std::vector<char> need(Bj, j == 0 ? 0 : 1);
    if ((err = run_stages(c, bk_network(Bj), seqs, lvl, need, dry, st, nprod, prog))) return err;
    if (j == 0) {
      lo = std::min(lo, min_level(lvl));
      if (!dry)
        for (uint32_t ch = 0; ch < chunks; ++ch)
          for (uint32_t t = 0; t < Bj; ++t) {
            if (prog) {
              prog->product(seqs[ch].cur_s[t], nullptr, nullptr, h[(size_t)ch * L + t]);
              ++prog->group;
              continue;
            }
            HIPCK_RET(hipMemcpyAsync(h[(size_t)ch * L + t], seqs[ch].cur_s[t],
                                     (size_t)2 * out_level * c->n * 8, hipMemcpyDeviceToDevice,
                                     st));
          }
      continue;
    }
    std::map<uint32_t, std::vector<uint32_t>> by_level;
    for (uint32_t t = 0; t < Bj; ++t) by_level[std::min(lvl[t], lvl_sum[j - 1])].push_back(t);
    for (const auto& kv : by_level) {
      const uint32_t l = kv.first;
      if (l < 2) return fail(FESC_ERR_LEVEL, "affine scan needs more levels than the input has");
      lo = std::min(lo, l - 1);
      if (nprod) *nprod += kv.second.size();
      if (dry) continue;
      std::vector<const uint64_t*> xs, ys, adds;
      std::vector<uint64_t*> outs;
      for (uint32_t ch = 0; ch < chunks; ++ch)
        for (uint32_t t : kv.second) {
          xs.push_back(seqs[ch].cur_a[t]);
          ys.push_back(carry[ch].cur_s[j - 1]);
          adds.push_back(seqs[ch].cur_s[t]);
          outs.push_back(h[(size_t)ch * L + (size_t)j * block + t]);
        }
      if (prog) {
        for (size_t i = 0; i < xs.size(); ++i) prog->product(xs[i], ys[i], adds[i], outs[i]);
        ++prog->group;
      } else if ((err = op_prod_rescale_many(c, (uint32_t)xs.size(), xs.data(), ys.data(),
                                             outs.data(), adds.data(), l, out_level, st))) {
        return err;
      }
    }
  }
  *min_out = lo;
  return FESC_OK;
}

size_t affine_scan_program(uint32_t L, uint32_t chunks, bool states_only, uint32_t level,
                           uint64_t* words, size_t cap, int* err) {
  // placeholder addresses as for the resident program; the scan is in place
  const uint64_t A0 = 1u << 24, S0 = 2u << 24;
  std::vector<uint64_t*> a((size_t)chunks * L), s((size_t)chunks * L);
  for (size_t i = 0; i < a.size(); ++i) {
    a[i] = reinterpret_cast<uint64_t*>((uintptr_t)(A0 + i));
    s[i] = reinterpret_cast<uint64_t*>((uintptr_t)(S0 + i));
  }
  Program prog;
  uint32_t lo;
  *err = scan_in_place(nullptr, a.data(), s.data(), L, chunks, level, states_only, &lo, nullptr,
                       &prog);
  if (words)
    for (size_t i = 0; i < prog.words.size() && i < 5 * cap; ++i) words[i] = prog.words[i];
  return prog.words.size() / 5;
}

size_t affine_scan_resident_program(uint32_t L, uint32_t block, uint32_t level, uint64_t* words,
                                    size_t cap, int* err) {
  // placeholder addresses (never dereferenced): inputs a, s, outputs h and the
  // workspace each get their own range
  const uint64_t A0 = 1u << 24, S0 = 2u << 24, H0 = 3u << 24, WS0 = 4u << 24;
  std::vector<const uint64_t*> a(L), s(L);
  std::vector<uint64_t*> h(L);
  for (uint32_t k = 0; k < L; ++k) {
    a[k] = reinterpret_cast<const uint64_t*>((uintptr_t)(A0 + k));
    s[k] = reinterpret_cast<const uint64_t*>((uintptr_t)(S0 + k));
    h[k] = reinterpret_cast<uint64_t*>((uintptr_t)(H0 + k));
  }
  Program prog;
  uint32_t lo;
  *err = resident(nullptr, a.data(), s.data(), L, 1, block, h.data(), level, 1,
                  reinterpret_cast<uint64_t*>((uintptr_t)WS0), false, &lo, nullptr, nullptr,
                  &prog);
  if (words)
    for (size_t i = 0; i < prog.words.size() && i < 5 * cap; ++i) words[i] = prog.words[i];
  return prog.words.size() / 5;
}

int op_affine_scan_resident_level(Context* c, uint32_t L, uint32_t block, uint32_t level,
                                  uint32_t* out_level, uint64_t* products) {
  uint64_t k = 0;
  int err = resident(c, nullptr, nullptr, L, 1, block, nullptr, level, 0, nullptr, true,
                     out_level, nullptr, &k);
  if (products) *products = k;
  return err;
}

int op_affine_scan_resident(Context* c, const uint64_t* const* a, const uint64_t* const* s,
                            uint32_t L, uint32_t chunks, uint32_t block, uint64_t* const* h,
                            uint32_t level, uint64_t* ws, uint32_t* out_level, hipStream_t st) {
  uint32_t lo;
  int err;
  if ((err = op_affine_scan_resident_level(c, L, block, level, &lo, nullptr))) return err;
  uint32_t got;
  if ((err = resident(c, a, s, L, chunks, block, h, level, lo, ws, false, &got, st))) return err;
  *out_level = lo;
  return FESC_OK;
}

}  // namespace fesc
