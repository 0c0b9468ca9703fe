// Eviction planning: which units to evict, in what order, and which restore
// path each evicted KV chunk takes.
//
// The paper balances its two restore paths (in-memory decompression and
// storage reads) by giving each increment of eviction to the path that keeps
// both finishing together, with weight layers restricted to one of the paths
// (Sec. 4.3, hybrid swap and balance preservation), and evicts in
// backward-out order (Sec. 4.4).  On this engine the two paths are the host
// link (swap: weights and KV chunks) and GPU recompute (drop: KV chunks
// only), so the same structure applies with one change: the cost of
// recomputing a chunk is not a fixed per-unit time.  Dropping chunk c at
// layer l pulls the rows of c through every layer up to l (they are in R_l'
// for all l' <= l), so its marginal cost depends on what else of column c is
// dropped.  The balanced placement therefore prices each candidate with the
// restore's exact FLOP count for the plan so far.
//
// Work model (integers, the restore path's own arithmetic):
//   R_l = {p < N : column(p) dropped at some l' >= l} U {N..S-1} U {S-1},
//   D_l = {p < N : column(p) dropped at l} U {N..S-1},
//   Q_l = R_{l+1} (l < L-1), {S-1} (l = L-1),
//   F_l = 2|Q_l| d 2dq + 2|D_l| d 2dkv + 2|Q_l| 3 d ff + 4 dq sum_{p in Q_l} (p+1).
// Time model (the restore's own schedule): the link copies forward-in, layer
// by layer (the weight unit, then the swapped chunks), so layer l's units
// have all arrived at A_l = (bytes of layers 0..l) / link rate; layer l's
// compute starts when layer l-1 is done and its units have arrived:
//   end_l = max(end_{l-1}, A_l) + F_l / recompute rate,  TTFT ~ end_{L-1}.
// A KV chunk goes to recompute when that gives the smaller end_{L-1}, else
// to the link (ties: link).  Times are exact integers in units of
// 1 / (link rate x recompute rate) seconds (rates rounded to whole bytes/s
// and FLOP/s, 128-bit arithmetic).
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/mz.h"
#include "mz_internal.h"

namespace {

typedef __int128 i128;

struct PlanError {
  mz_status st;
  const char* msg;
};

// splitmix64 (Steele, Lea and Flood, OOPSLA 2014, with the published
// constants): the random-out order's generator.
uint64_t splitmix64(uint64_t& x) {
  uint64_t z = (x += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

struct Work {
  int L, nc, C, N, P, S;
  int64_t d, dq, dkv, ff;
  std::vector<int64_t> rows, psum;   // per column: context rows, sum of (p+1)
  std::vector<int> md;               // per column: deepest layer that drops it, -1 if none
  std::vector<int64_t> drop_rows;    // per layer: context rows of columns dropped there
  int64_t prompt_psum = 0;           // sum of (p+1) over the prompt positions

  Work(const mz_model_cfg& c, int n_ctx, int n_prompt)
      : L(c.n_layers), nc((n_ctx + c.chunk_tokens - 1) / c.chunk_tokens), C(c.chunk_tokens), N(n_ctx),
        P(n_prompt), S(n_ctx + n_prompt), d(c.d_model), dq((int64_t)c.n_q_heads * c.head_dim),
        dkv((int64_t)c.n_kv_heads * c.head_dim), ff(c.d_ffn) {
    rows.resize(nc);
    psum.resize(nc);
    for (int k = 0; k < nc; ++k) {
      const int64_t p0 = (int64_t)k * C, n = std::min<int64_t>(C, N - p0);
      rows[k] = n;
      psum[k] = n * (p0 + 1) + n * (n - 1) / 2;
    }
    md.assign(nc, -1);
    drop_rows.assign(L, 0);
    for (int64_t p = N; p < S; ++p) prompt_psum += p + 1;
  }

  // |R_l| and sum_{p in R_l} (p+1)
  void rset(int l, int64_t& n, int64_t& ps) const {
    n = P;
    ps = prompt_psum;
    for (int k = 0; k < nc; ++k)
      if (md[k] >= l) {
        n += rows[k];
        ps += psum[k];
      }
    if (P == 0 && nc > 0 && md[nc - 1] < l) {   // the last position joins every R_l
      n += 1;
      ps += S;
    }
  }

  int64_t layer_flops(int l) const {
    int64_t nq, aq;
    if (l + 1 < L) {
      rset(l + 1, nq, aq);
    } else {
      nq = 1;
      aq = S;
    }
    const int64_t nd = drop_rows[l] + P;
    return 2 * nq * d * 2 * dq + 2 * nd * d * 2 * dkv + 2 * nq * 3 * d * ff + 4 * dq * aq;
  }
  int64_t flops() const {
    int64_t f = 0;
    for (int l = 0; l < L; ++l) f += layer_flops(l);
    return f;
  }
  // end of the last layer in units of 1 / (BW * RF) s, given the bytes each
  // layer brings over the link
  i128 pipeline_end(const std::vector<int64_t>& layer_bytes, i128 BW, i128 RF) const {
    i128 arrive = 0, end = 0;
    for (int l = 0; l < L; ++l) {
      arrive += (i128)layer_bytes[l] * RF;
      end = std::max(end, arrive) + (i128)layer_flops(l) * BW;
    }
    return end;
  }

  void drop(int l, int k) {
    md[k] = std::max(md[k], l);
    drop_rows[l] += rows[k];
  }
  void undrop(int l, int k, int old_md) {
    md[k] = old_md;
    drop_rows[l] -= rows[k];
  }
};

}  // namespace

extern "C" {

mz_status mz_plan_evict(const mz_model_cfg* cfg, const mz_evict_request* req, uint8_t* kv_state,
                        uint8_t* w_state, double* est) {
  try {
    if (!cfg || !req || !kv_state || !w_state) throw PlanError{MZ_EINVAL, "NULL pointer"};
    const mz_model_cfg& c = *cfg;
    if (c.n_layers < 1 || c.chunk_tokens < 1 || req->n_ctx < 1 || req->n_prompt < 0)
      throw PlanError{MZ_EINVAL, "bad sizes"};
    Work w(c, req->n_ctx, req->n_prompt);
    const int L = w.L, nc = w.nc;
    if (req->n_kv_evict < 0 || req->n_kv_evict > L * nc) throw PlanError{MZ_EINVAL, "n_kv_evict out of range"};
    if (req->n_w_evict < 0 || req->n_w_evict > L) throw PlanError{MZ_EINVAL, "n_w_evict out of range"};
    if (req->placement == MZ_PLACE_BALANCED && !(req->link_bytes_per_s >= 1.0 && req->recompute_flops_per_s >= 1.0))
      throw PlanError{MZ_EINVAL, "balanced placement needs positive rates"};

    // eviction order over the KV units (layer, column)
    std::vector<std::pair<int, int>> seq;
    seq.reserve((size_t)L * nc);
    switch (req->order) {
      case MZ_ORDER_BACKWARD_OUT:
        for (int l = L - 1; l >= 0; --l)
          for (int k = nc - 1; k >= 0; --k) seq.push_back({l, k});
        break;
      case MZ_ORDER_FORWARD_OUT:
        for (int l = 0; l < L; ++l)
          for (int k = 0; k < nc; ++k) seq.push_back({l, k});
        break;
      case MZ_ORDER_TOKEN_ALIGNED:
        for (int k = nc - 1; k >= 0; --k)
          for (int l = L - 1; l >= 0; --l) seq.push_back({l, k});
        break;
      case MZ_ORDER_RANDOM_OUT: {
        for (int l = L - 1; l >= 0; --l)
          for (int k = nc - 1; k >= 0; --k) seq.push_back({l, k});
        uint64_t x = req->seed;
        for (size_t i = seq.size() - 1; i > 0; --i) {   // Fisher-Yates
          const size_t j = (size_t)(splitmix64(x) % (uint64_t)(i + 1));
          std::swap(seq[i], seq[j]);
        }
        break;
      }
      default:
        throw PlanError{MZ_EINVAL, "unknown order"};
    }

    memset(kv_state, MZ_RES, (size_t)L * nc);
    memset(w_state, MZ_RES, (size_t)L);
    const int64_t slot = mzrt::kv_slot_bytes(c), unit = mzrt::weight_unit_bytes(c);
    // link bytes of a swapped chunk: compressed when the codec is on and the
    // chunk is full (n halves -> n + n/16 bytes), else the raw slot
    const int64_t comp = slot / 2 + slot / 32;
    auto chunk_link_bytes = [&](int k) {
      return req->kv_codec && (int64_t)(k + 1) * c.chunk_tokens <= req->n_ctx ? comp : slot;
    };
    int64_t link_bytes = 0;
    std::vector<int64_t> layer_bytes(L, 0);
    // weight units ride the link: the last layers, or the first for forward-out
    for (int i = 0; i < req->n_w_evict; ++i) {
      const int l = req->order == MZ_ORDER_FORWARD_OUT ? i : L - 1 - i;
      w_state[l] = MZ_SWAP;
      link_bytes += unit;
      layer_bytes[l] += unit;
    }
    const i128 BW = (i128)(int64_t)(req->link_bytes_per_s + 0.5);
    const i128 RF = (i128)(int64_t)(req->recompute_flops_per_s + 0.5);
    int64_t f_cur = w.flops();
    for (int r = 0; r < req->n_kv_evict; ++r) {
      const int l = seq[r].first, k = seq[r].second;
      bool drop = false;
      switch (req->placement) {
        case MZ_PLACE_ALL_SWAP: drop = false; break;
        case MZ_PLACE_ALL_DROP: drop = true; break;
        case MZ_PLACE_INTERLEAVE_2_1: drop = r % 3 == 2; break;
        case MZ_PLACE_BALANCED: {
          layer_bytes[l] += chunk_link_bytes(k);
          const i128 if_swap = w.pipeline_end(layer_bytes, BW, RF);
          layer_bytes[l] -= chunk_link_bytes(k);
          const int old = w.md[k];
          w.drop(l, k);
          const i128 if_drop = w.pipeline_end(layer_bytes, BW, RF);
          w.undrop(l, k, old);
          drop = if_drop < if_swap;
          break;
        }
        default:
          throw PlanError{MZ_EINVAL, "unknown placement"};
      }
      if (drop) {
        kv_state[(size_t)l * nc + k] = MZ_DROP;
        w.drop(l, k);
        f_cur = w.flops();
      } else {
        kv_state[(size_t)l * nc + k] = MZ_SWAP;
        link_bytes += chunk_link_bytes(k);
        layer_bytes[l] += chunk_link_bytes(k);
      }
    }
    if (est) {
      est[0] = (double)link_bytes;
      est[1] = (double)f_cur;
      est[2] = BW > 0 ? (double)link_bytes / (double)BW : 0.0;
      est[3] = RF > 0 ? (double)f_cur / (double)RF : 0.0;
      est[4] = BW > 0 && RF > 0 ? (double)w.pipeline_end(layer_bytes, BW, RF) / ((double)BW * (double)RF) : 0.0;
    }
    return MZ_OK;
  } catch (const PlanError& e) {
    mzrt::set_error(e.msg);
    return e.st;
  }
}

// Size-driven eviction: the hybrid-swap state machine (paper Alg. 1) over
// the two restore paths, one unit at a time, rearmost first.  Totals are
// kept in units of 1 / (BW * RF) seconds: link bytes * RF, recompute FLOPs *
// BW.  Every decision reads only the current unit states, so a sequence of
// calls takes the same units as one call asking for their sum.
mz_status mz_plan_evict_size(const mz_model_cfg* cfg, int32_t n_ctx, const mz_evict_size_request* req,
                             uint8_t* kv_state, uint8_t* w_state, int32_t* order, int32_t* stage,
                             int32_t* n_evicted, double* info) {
  try {
    if (!cfg || !req || !kv_state || !w_state) throw PlanError{MZ_EINVAL, "NULL pointer"};
    const mz_model_cfg& c = *cfg;
    if (c.n_layers < 1 || c.chunk_tokens < 1 || n_ctx < 1 || req->n_prompt < 0 || req->bytes < 0)
      throw PlanError{MZ_EINVAL, "bad sizes"};
    if (req->n_w_total < 0 || req->n_w_total > c.n_layers) throw PlanError{MZ_EINVAL, "n_w_total out of range"};
    if (!(req->link_bytes_per_s >= 1.0 && req->recompute_flops_per_s >= 1.0))
      throw PlanError{MZ_EINVAL, "size-driven eviction needs positive rates"};
    if (req->rule != MZ_SIZE_RULE_PAPER && req->rule != MZ_SIZE_RULE_TOTAL)
      throw PlanError{MZ_EINVAL, "unknown size rule"};
    Work w(c, n_ctx, req->n_prompt);
    const int L = w.L, nc = w.nc, total = L * nc;
    for (int u = 0; u < total; ++u)
      if (kv_state[u] > MZ_DROP) throw PlanError{MZ_EINVAL, "invalid kv_state entry"};
    for (int l = 0; l < L; ++l)
      if (w_state[l] > MZ_DROP) throw PlanError{MZ_EINVAL, "invalid w_state entry"};
    const i128 BW = (i128)(int64_t)(req->link_bytes_per_s + 0.5);
    const i128 RF = (i128)(int64_t)(req->recompute_flops_per_s + 0.5);
    const int64_t slot = mzrt::kv_slot_bytes(c), unit = mzrt::weight_unit_bytes(c);
    const int64_t comp = slot / 2 + slot / 32;
    auto chunk_link_bytes = [&](int k) {
      return req->kv_codec && (int64_t)(k + 1) * c.chunk_tokens <= n_ctx ? comp : slot;
    };
    const int64_t F0 = w.flops();

    // backward-out order over every chunk; weights rearmost first
    std::vector<std::pair<int, int>> seq;
    seq.reserve(total);
    for (int l = L - 1; l >= 0; --l)
      for (int k = nc - 1; k >= 0; --k) seq.push_back({l, k});

    // threshold T and the KV_AND_W pairing
    const bool paper = req->rule == MZ_SIZE_RULE_PAPER;
    int64_t T = 0, k_pair = 0;
    if (paper) {
      // k = floor(t_W / t_d): t_W = unit / BW, t_d = (front-most chunk's FLOPs) / RF
      Work t(c, n_ctx, req->n_prompt);
      t.drop(0, 0);
      const i128 den = (i128)(t.flops() - F0) * BW;
      const i128 kk = den > 0 ? (i128)unit * RF / den : 0;
      k_pair = kk > (i128)INT32_MAX ? (int64_t)INT32_MAX : (int64_t)kk;
      T = (int64_t)req->n_w_total * k_pair;
    } else {
      // the front-most chunks whose recompute fits the reload of all
      // evictable weight layers
      const i128 budget = (i128)req->n_w_total * unit * RF;
      auto tail_fits = [&](int n) {
        Work t(c, n_ctx, req->n_prompt);
        for (int i = total - n; i < total; ++i) t.drop(seq[i].first, seq[i].second);
        return (i128)(t.flops() - F0) * BW <= budget;
      };
      int lo = 0, hi = total;   // the cost grows with n
      while (lo < hi) {
        const int mid = (lo + hi + 1) / 2;
        if (tail_fits(mid)) lo = mid; else hi = mid - 1;
      }
      T = lo;
    }

    // current state
    int64_t link = 0;
    int n_kv = 0, n_w = 0;
    for (int l = 0; l < L; ++l)
      for (int k = 0; k < nc; ++k) {
        const uint8_t st = kv_state[(size_t)l * nc + k];
        if (st == MZ_RES) ++n_kv;
        else if (st == MZ_SWAP) link += chunk_link_bytes(k);
        else w.drop(l, k);
      }
    for (int l = 0; l < L; ++l) {
      if (w_state[l] != MZ_RES) link += unit;
      else if (l >= L - req->n_w_total) ++n_w;
    }
    int64_t F = w.flops();
    size_t kv_cur = 0;
    int w_cur = L - 1;
    auto next_kv = [&]() {
      while (kv_state[(size_t)seq[kv_cur].first * nc + seq[kv_cur].second] != MZ_RES) ++kv_cur;
      return seq[kv_cur];
    };
    auto next_w = [&]() {
      while (w_state[w_cur] != MZ_RES) --w_cur;
      return w_cur;
    };
    // paper rule: the weight layers taken in KV_AND_W still cover chunks not
    // yet taken (the stage began at N_KV = min(T, all chunks))
    auto owed = [&]() {
      return paper && std::min<int64_t>(T, total) - n_kv < k_pair * (int64_t)(req->n_w_total - n_w);
    };
    auto stage_now = [&]() {
      if (n_kv > T) return (int)MZ_STAGE_KV_ONLY;
      if (n_kv > 0 && (n_w > 0 || owed())) return (int)MZ_STAGE_KV_AND_W;
      if (n_kv > 0) return (int)MZ_STAGE_KV_ONLY;
      if (n_w > 0) return (int)MZ_STAGE_W_ONLY;
      return (int)MZ_STAGE_EXHAUSTED;
    };

    int64_t released = 0;
    int n_out = 0;
    int st = stage_now();
    while (released < req->bytes && st != MZ_STAGE_EXHAUSTED) {
      int unit_id;
      if (st == MZ_STAGE_W_ONLY) {
        const int l = next_w();
        w_state[l] = MZ_DROP;
        link += unit;
        --n_w;
        released += unit;
        unit_id = total + l;
      } else if (st == MZ_STAGE_KV_AND_W && paper && n_w > 0 && !owed()) {
        // the paper's pairing: a weight layer, then the k chunks its reload covers
        const int l = next_w();
        w_state[l] = MZ_DROP;
        link += unit;
        --n_w;
        released += unit;
        unit_id = total + l;
      } else {
        const auto lk = next_kv();
        const int l = lk.first, k = lk.second, old = w.md[k];
        w.drop(l, k);
        const int64_t Fd = w.flops();
        const i128 rec_with = (i128)(Fd - F0) * BW;
        bool drop, take_weight = false;
        if (st == MZ_STAGE_KV_ONLY) {
          drop = rec_with < (i128)(link + chunk_link_bytes(k)) * RF;
        } else if (paper) {
          drop = true;
        } else {
          drop = rec_with <= (i128)link * RF;
          take_weight = !drop;
        }
        if (take_weight) {
          w.undrop(l, k, old);
          const int lw = next_w();
          w_state[lw] = MZ_DROP;
          link += unit;
          --n_w;
          released += unit;
          unit_id = total + lw;
        } else {
          if (drop) {
            F = Fd;
            kv_state[(size_t)l * nc + k] = MZ_DROP;
          } else {
            w.undrop(l, k, old);
            kv_state[(size_t)l * nc + k] = MZ_SWAP;
            link += chunk_link_bytes(k);
          }
          --n_kv;
          released += slot;
          unit_id = l * nc + k;
        }
      }
      if (order) order[n_out] = unit_id;
      if (stage) stage[n_out] = st;
      ++n_out;
      st = stage_now();
    }
    if (n_evicted) *n_evicted = n_out;
    if (info) {
      info[0] = (double)released;
      info[1] = (double)T;
      info[2] = (double)st;
      info[3] = (double)link / (double)BW;
      info[4] = (double)(F - F0) / (double)RF;
      info[5] = (double)n_kv;
      info[6] = (double)n_w;
      info[7] = released >= req->bytes ? 1.0 : 0.0;
    }
    return MZ_OK;
  } catch (const PlanError& e) {
    mzrt::set_error(e.msg);
    return e.st;
  }
}

}  // extern "C"
