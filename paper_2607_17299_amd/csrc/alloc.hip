// Paged-KV bookkeeping kernels: free stack, reference counts, block tables,
// reserve / commit / rollback / fork / free, and the verify-step setup that
// reserves draft slots and builds the step's row metadata and attention work list.
//
// Every bookkeeping kernel runs as ONE workgroup of 1024 threads, so its effect
// is a deterministic function of its inputs (no cross-workgroup atomics).
// Policy: pops for batch entries in ascending order, logical pages ascending;
// pushes in descending entry order, logical pages descending -- a reserve
// followed by a discard restores the stack exactly.
#include "kernels.h"

namespace {

constexpr int kBT = 1024;

// Exclusive scan of one int per thread over the block; *total receives the sum.
__device__ int block_excl_scan(int v, int* sh, int* total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6, nw = blockDim.x >> 6;
  int x = v;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  __syncthreads();
  if (lane == 63) sh[w] = x;
  __syncthreads();
  int off = 0, tot = 0;
  for (int i = 0; i < nw; ++i) {
    if (i < w) off += sh[i];
    tot += sh[i];
  }
  *total = tot;
  __syncthreads();
  return off + x - v;
}

__global__ void k_pool_init(PoolDev p) {
  const int64_t n_tab = (int64_t)p.max_seqs * p.max_pages;
  const int64_t n_all = n_tab > p.num_pages ? n_tab : (int64_t)p.num_pages;
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n_all;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (i < n_tab) p.table[i] = -1;
    if (i < p.num_pages) {
      p.stack[i] = p.num_pages - 1 - (int32_t)i;
      p.refcount[i] = 0;
    }
    if (i < p.max_seqs) {
      p.held[i] = 0;
      p.base[i] = 0;
    }
    if (i == 0) {
      p.scalars[0] = p.num_pages;
      p.scalars[1] = 0;
      p.scalars[2] = 0;
    }
  }
}

// Pop `need` pages for entry (seq s) after `off` earlier pops of this call.
__device__ void pop_pages(const PoolDev& p, int s, int need, int off, int fc) {
  const int h = p.held[s];
  int32_t* row = p.table + (int64_t)s * p.max_pages;
  for (int j = 0; j < need; ++j) {
    const int page = p.stack[fc - 1 - (off + j)];
    row[h + j] = page;
    p.refcount[page] = 1;
  }
}

// Grow sequences to `target` pages (mode 0: alloc, targets from n_tokens;
// mode 1: prefill, targets from ctx + n_new).  One thread per entry, n <= 1024.
__global__ void __launch_bounds__(kBT) k_grow(PoolDev p, int n, const int32_t* seq_ids,
                                              const int32_t* a, const int32_t* b, int mode) {
  __shared__ int sh[16];
  __shared__ int s_fail;
  const int t = threadIdx.x;
  int s = 0, need = 0, target = 0;
  if (t < n) {
    s = seq_ids[t];
    const int tokens = mode == 0 ? a[t] : a[t] + b[t];
    target = cdiv_i(tokens, p.page_size);
    need = max(0, target - p.held[s]);
  }
  int total;
  const int off = block_excl_scan(need, sh, &total);
  const int fc = p.scalars[0];
  if (t == 0) s_fail = total > fc;
  __syncthreads();
  if (s_fail) {
    if (t == 0) p.scalars[1] |= ERR_NO_PAGES;
    return;
  }
  if (t < n) {
    pop_pages(p, s, need, off, fc);
    p.held[s] += need;
    p.base[s] = p.held[s];
  }
  __syncthreads();
  if (t == 0) p.scalars[0] = fc - total;
}

// Verify-step setup: reserve pages for ctx + draft_len + 1 slots per request,
// then build the padded row layout (row b*(k+1)+i = request b, token i) and the
// attention work list (one item per `chunk` keys of each request).  With tree
// drafts (k_max + 1 <= 32) token i is tree node i.
__global__ void __launch_bounds__(kBT) k_verify_setup(PoolDev p, VerifySetupArgs a, StepMeta m) {
  __shared__ int sh[16];
  __shared__ int s_fail;
  __shared__ int s_ctx[kBT], s_dl[kBT];
  __shared__ int s_pg0[kBT], s_nch[kBT], s_seq[kBT], s_shr[kBT], s_noff[kBT], s_run[kBT];
  __shared__ int s_lead[kBT], s_np[kBT], s_mis[kBT];
  constexpr int kHash = 2 * kBT;  // open-addressing table of the step's ids
  __shared__ int s_hash[kHash];
  const int t = threadIdx.x;
  const int kp1 = a.k_max + 1;
  __shared__ int s_bad, s_dup;
  if (t == 0) {
    s_bad = 0;
    s_dup = 0;
  }
  // the attention launches of this step start their work counters at zero
  if (t < 8) a.unit_ctr[t] = 0;
  for (int i = t; i < kHash; i += kBT) s_hash[i] = -1;
  __syncthreads();
  int s = 0, need = 0, ctx = 0, dl = 0, hb = 0;
  if (t < a.B) {
    s = a.seq_ids[t];
    ctx = a.ctx_lens[t];
    dl = a.draft_lens ? a.draft_lens[t] : a.k_max;
    dl = min(max(dl, 0), a.k_max);
    // a bad id, a negative length or a request beyond its block-table row
    // fails the whole step (no page moves, no row is active)
    if (s < 0 || s >= p.max_seqs || ctx < 0 ||
        cdiv_i(ctx + dl + 1, p.page_size) > p.max_pages) {
      s = 0;
      ctx = 0;
      atomicOr(&s_bad, 1);
    } else {
      // two entries with one id would pop into the same block-table row:
      // insert the id (linear probing; B <= kBT ids never fill the table)
      unsigned hsh = ((unsigned)s * 2654435761u) >> 21;
      for (int probe = 0; probe < kHash; ++probe) {
        const int prev = atomicCAS(&s_hash[hsh], -1, s);
        if (prev == -1) break;
        if (prev == s) {
          atomicOr(&s_dup, 1);
          break;
        }
        hsh = (hsh + 1) & (kHash - 1);
      }
      hb = p.held[s];
      need = max(0, cdiv_i(ctx + dl + 1, p.page_size) - hb);
    }
  }
  int total;
  const int off = block_excl_scan(need, sh, &total);  // (its barriers order the inserts)
  const int fc = p.scalars[0];
  if (t == 0) {
    s_fail = total > fc || s_bad || s_dup;
    if (s_bad) atomicOr(&p.scalars[1], ERR_BAD_TOKEN);
    if (s_dup) atomicOr(&p.scalars[1], ERR_DUP_SEQ);
  }
  __syncthreads();
  const bool fail = s_fail;
  if (t < a.B) {
    if (!fail) {
      pop_pages(p, s, need, off, fc);
      p.held[s] = hb + need;
      p.base[s] = hb;
    }
    s_ctx[t] = ctx;
    s_dl[t] = fail ? -1 : dl;
    m.req_seq[t] = s;
    m.req_pos0[t] = ctx;
    m.req_ntok[t] = fail ? 0 : dl + 1;
    m.req_row0[t] = t * kp1;
  }
  // attention items: chunks of the keys visible to the request's last row.
  // Longer chunks mean fewer partials to write and merge and fewer unit
  // changes; they are used when the batch still has enough items for the grid
  // and no sequences share pages (siblings that read a shared chunk at the same
  // time find it in L2 more often when the chunks are short).
  int n2;
  (void)block_excl_scan((t < a.B && !fail) ? cdiv_i(ctx + dl + 1, 2 * a.chunk) : 0, sh, &n2);
  const int chunk = n2 >= a.items_double && !a.cascade ? 2 * a.chunk : a.chunk;
  const int nch = (t < a.B && !fail) ? cdiv_i(ctx + dl + 1, chunk) : 0;
  int n_items;
  const int ioff = block_excl_scan(nch, sh, &n_items);
  if (t < a.B) {
    m.seg_begin[t] = ioff;
    m.seg_count[t] = nch;
    m.seg_req[t] = t;
    m.seg_rb[t] = 0;
    for (int c = 0; c < nch; ++c) m.items[ioff + c] = make_int4(t, 0, c, 0);
    s_pg0[t] = (!fail && ctx > 0) ? p.table[(int64_t)s * p.max_pages] : -1 - t;
    s_nch[t] = nch;
    s_seq[t] = s;
    s_shr[t] = 0x7fffffff;
  }
  __syncthreads();
  // Groups: consecutive requests whose first page is the same physical page
  // (forked siblings).  The keys a group shares are the whole pages every
  // member has in common with the first member, within every member's context
  // (so visible to every row of the step).
  int L = t, g = 1;
  bool regular = true;
  if (t < a.B) {
    while (L > 0 && s_pg0[L - 1] == s_pg0[t]) --L;
    while (L + g < a.B && s_pg0[L + g] == s_pg0[L]) {
      regular = regular && s_nch[L + g] == s_nch[L];
      ++g;
    }
    s_lead[t] = L;
    s_np[t] = (g > 1 && nch > 0) ? min(s_ctx[t], s_ctx[L]) / p.page_size : -1;
    s_mis[t] = max(s_np[t], 0);
  }
  __syncthreads();
  // first page (below np) where a member's block table differs from the first
  // member's: all threads compare one request's pages at a time
  for (int q = 0; q < a.B; ++q) {
    const int np = s_np[q];
    if (np <= 0) continue;
    const int32_t* rb = p.table + (int64_t)s_seq[q] * p.max_pages;
    const int32_t* rl = p.table + (int64_t)s_seq[s_lead[q]] * p.max_pages;
    for (int c = t; c < np; c += kBT)
      if (rb[c] != rl[c]) atomicMin(&s_mis[q], c);
  }
  __syncthreads();
  if (t < a.B && s_np[t] >= 0) atomicMin(&s_shr[L], s_mis[t] * p.page_size);
  __syncthreads();
  // Shared-prefix units: the whole attention chunks a group shares are attended
  // once per run of consecutive members whose live rows (G per token) fit one
  // row block together; the unit writes every member's partial.  The first
  // member of a run owns it (item .w = members); the others' items for those
  // chunks are never scheduled (.w = -1).  Ordinary items keep .w = 0.
  const int RBs = a.rb;
  if (t < a.B && a.cascade && L == t && g > 1 && nch > 0 && s_shr[t] >= chunk) {
    int j0 = 0, rows = 0;
    for (int jj = 0; jj < g; ++jj) {
      const int rj = a.G * (s_dl[t + jj] + 1);
      if (jj > j0 && rows + rj > RBs) {
        s_run[t + j0] = jj - j0;
        j0 = jj;
        rows = 0;
      }
      rows += rj;
      s_run[t + jj] = 0;
    }
    s_run[t + j0] = g - j0;
  }
  __syncthreads();
  int nsc = 0;
  if (t < a.B && a.cascade && g > 1 && nch > 0 && s_shr[L] >= chunk) nsc = min(s_shr[L] / chunk, nch);
  const int j = t - L;
  const int run = nsc > 0 ? s_run[t] : 0;  // members of the run this request owns (0: not an owner)
  if (t < a.B && nsc > 0)
    for (int c = 0; c < nsc; ++c) m.items[ioff + c].w = run > 0 ? run : -1;
  const int n_mine = (t < a.B) ? nch - nsc + (run > 0 ? nsc : 0) : 0;
  int n_units;
  const int noff = block_excl_scan(n_mine, sh, &n_units);
  if (t < a.B) s_noff[t] = noff;
  // A batch without forked siblings takes every request's whole chunks first,
  // in request order, then the partial last chunks, longest first: the
  // persistent grid then ends on its shortest units (s_mis is free by now and
  // holds each request's partial length).
  __shared__ int s_grp;
  if (t == 0) s_grp = 0;
  __syncthreads();
  if (t < a.B && g > 1) s_grp = 1;  // every writer stores 1
  const int len = (t < a.B && nch > 0) ? ctx + dl + 1 : 0;
  const int n_whole = len / chunk, rem = len % chunk;
  if (t < a.B) s_mis[t] = rem;
  __syncthreads();
  const bool lpt = s_grp == 0;
  int n_whole_all;
  const int woff = block_excl_scan(lpt ? n_whole : 0, sh, &n_whole_all);
  // Work order.  A group without shared units whose members have equal chunk
  // counts gets its items interleaved chunk-major (the members read a shared
  // chunk at the same time, so later readers find it in cache); otherwise
  // request order, a run's shared units first.
  if (t < a.B && nch > 0) {
    // slot o of the order gets chunk c of this request (and its descriptor)
    auto put = [&](int o, int c) {
      m.order[o] = ioff + c;
      const int wc = c < nsc ? (run > 0 ? run : -1) : 0;
      m.udesc[2 * o] = make_int4(ioff + c, t, c, (dl + 1) << 16);  // first token 0, dl + 1 rows' tokens
      m.udesc[2 * o + 1] = make_int4(wc, s, ctx, t * kp1);
    };
    if (lpt) {
      for (int c = 0; c < n_whole; ++c) put(woff + c, c);
      if (rem > 0) {
        int rank = 0;  // partial chunks longer than this one, ties by request
        for (int q = 0; q < a.B; ++q) {
          const int rq = s_mis[q];
          rank += rq > rem || (rq == rem && q < t);
        }
        put(n_whole_all + rank, n_whole);
      }
    } else if (nsc == 0 && g > 1 && regular) {
      for (int c = 0; c < nch; ++c) put(s_noff[L] + c * g + j, c);
    } else {
      int o = noff;
      if (run > 0)
        for (int c = 0; c < nsc; ++c) put(o++, c);
      for (int c = nsc; c < nch; ++c) put(o++, c);
    }
  }
  if (t == 0) {
    m.n_items[0] = n_items;
    m.n_items[1] = n_units;
    m.n_items[2] = 0;
    m.n_items[3] = chunk;
    if (fail && !s_bad && !s_dup) p.scalars[1] |= ERR_NO_PAGES;
    if (!fail) p.scalars[0] = fc - total;
    p.scalars[2] = fail ? 1 : 0;  // the commit of a failed step changes nothing
  }
  __syncthreads();
  // rows: request b's token i sits in row b*(k_max+1)+i
  const int R = a.B * kp1;
  for (int r = t; r < R; r += blockDim.x) {
    const int b = r / kp1, i = r % kp1;
    const int dlb = s_dl[b];
    const bool act = i <= dlb;
    int tok = 0;
    if (act) tok = i == 0 ? a.last_tokens[b] : a.draft_tokens[(int64_t)b * a.k_max + i - 1];
    if (tok < 0 || tok >= a.vocab) {
      atomicOr(&p.scalars[1], ERR_BAD_TOKEN);
      tok = 0;
    }
    m.tok[r] = tok;
    m.active[r] = act ? 1 : 0;
    m.row_req[r] = b;
    const int slot = s_ctx[b] + min(i, max(dlb, 0));
    if (a.draft_parents) {
      // tree drafts: node i sits in slot ctx + i at position ctx + depth; its
      // mask holds the nodes of its root path.  A parent outside [0, i) is
      // flagged and read as i - 1, so the walk always ends.
      int depth = 0;
      uint32_t msk = 1u;
      if (act)
        for (int j = i; j > 0; ++depth) {
          msk |= 1u << j;
          int pj = a.draft_parents[(int64_t)b * a.k_max + j - 1];
          if (pj < 0 || pj >= j) {
            atomicOr(&p.scalars[1], ERR_BAD_PARENT);
            pj = j - 1;
          }
          j = pj;
        }
      m.pos[r] = s_ctx[b] + depth;
      m.kvpos[r] = slot;
      m.tmask[r] = msk;
    } else {
      m.pos[r] = slot;
    }
  }
}

// Commit: keep ctx + a + 1 tokens, push the step's pages beyond them
// (entries in descending order, logical pages descending).  After a verify
// step whose setup failed nothing changes.  Thread 0 then reports
// (commit_seq, free count) to the host-mapped word.
__global__ void __launch_bounds__(kBT) k_commit(PoolDev p, int B, const int32_t* seq_ids,
                                                int32_t* ctx_lens, const int32_t* accept,
                                                uint32_t commit_seq) {
  __shared__ int sh[16];
  __shared__ int s_skip;
  const int t = threadIdx.x;
  if (t == 0) s_skip = p.scalars[2];
  __syncthreads();
  if (s_skip) {
    if (t == 0) {
      p.scalars[2] = 0;
      __hip_atomic_store(p.report, ((unsigned long long)commit_seq << 32) | (uint32_t)p.scalars[0],
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }
    return;
  }
  const int rt = B - 1 - t;  // entry handled by this thread, so the scan runs descending
  int s = 0, h = 0, keep = 0, rel = 0, new_ctx = 0;
  bool ok = false;
  if (t < B) {
    s = seq_ids[rt];
    // the verify step accepted these ids; other ids (a different array than
    // the step's) are flagged and left alone
    ok = s >= 0 && s < p.max_seqs;
    if (!ok) atomicOr(&p.scalars[1], ERR_BAD_TOKEN);
  }
  if (ok) {
    h = p.held[s];
    const int ctx = ctx_lens[rt];
    const int cap = h * p.page_size;
    const int acc = min(max(accept[rt], -1), cap - ctx - 1);
    new_ctx = ctx + max(acc, -1) + 1;
    keep = min(h, max(p.base[s], cdiv_i(new_ctx, p.page_size)));
    rel = h - keep;
  }
  int total;
  const int off = block_excl_scan(rel, sh, &total);
  const int fc = p.scalars[0];
  if (ok) {
    int32_t* row = p.table + (int64_t)s * p.max_pages;
    for (int j = 0; j < rel; ++j) {
      const int page = row[h - 1 - j];
      p.stack[fc + off + j] = page;
      p.refcount[page] -= 1;
      row[h - 1 - j] = -1;
    }
    p.held[s] = keep;
    p.base[s] = keep;
    ctx_lens[rt] = new_ctx;
  }
  __syncthreads();
  if (t == 0) {
    p.scalars[0] = fc + total;
    __hip_atomic_store(p.report, ((unsigned long long)commit_seq << 32) | (uint32_t)(fc + total),
                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
  }
}

// Free sequences: entries in descending order; within one, logical pages
// descending; a page is pushed when its count drops to 0.
__global__ void __launch_bounds__(kBT) k_free(PoolDev p, int n, const int32_t* seq_ids) {
  __shared__ int sh[16];
  __shared__ int s_fc;
  if (threadIdx.x == 0) s_fc = p.scalars[0];
  __syncthreads();
  for (int e = n - 1; e >= 0; --e) {
    const int s = seq_ids[e];
    const int h = p.held[s];
    int32_t* row = p.table + (int64_t)s * p.max_pages;
    for (int c0 = 0; c0 < h; c0 += blockDim.x) {
      const int j = h - 1 - (c0 + threadIdx.x);  // descending logical page
      int page = -1, push = 0;
      if (j >= 0) {
        page = row[j];
        push = p.refcount[page] == 1;
      }
      int total;
      const int off = block_excl_scan(push, sh, &total);
      const int fc = s_fc;
      if (j >= 0) {
        p.refcount[page] -= 1;
        if (push) p.stack[fc + off] = page;
        row[j] = -1;
      }
      __syncthreads();
      if (threadIdx.x == 0) s_fc = fc + total;
      __syncthreads();
    }
    if (threadIdx.x == 0) {
      p.held[s] = 0;
      p.base[s] = 0;
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) p.scalars[0] = s_fc;
}

__global__ void k_fork(PoolDev p, int src, int dst, int npg) {
  const int32_t* rs = p.table + (int64_t)src * p.max_pages;
  int32_t* rd = p.table + (int64_t)dst * p.max_pages;
  for (int j = threadIdx.x; j < npg; j += blockDim.x) {
    const int page = rs[j];
    rd[j] = page;
    p.refcount[page] += 1;  // a sequence's pages are distinct: no two threads share one
  }
  if (threadIdx.x == 0) {
    p.held[dst] = npg;
    p.base[dst] = npg;
  }
}

// Copy [2][Hkv][n][D] keys/values of tokens pos0.. into the sequence's pages.
__global__ void k_kv_load(PoolDev p, KvGeom g, int seq, int layer, int pos0, int n,
                          const bf16_t* src) {
  const int64_t total = (int64_t)2 * g.n_kv_heads * n * g.head_dim;
  const int32_t* row = p.table + (int64_t)seq * p.max_pages;
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
       e += (int64_t)gridDim.x * blockDim.x) {
    const int d = (int)(e % g.head_dim);
    const int64_t r = e / g.head_dim;
    const int tkn = (int)(r % n);
    const int kvh = (int)((r / n) % g.n_kv_heads);
    const int kind = (int)(r / ((int64_t)n * g.n_kv_heads));
    const int pos = pos0 + tkn;
    const int page = row[pos / p.page_size], slot = pos % p.page_size;
    bf16_t* base = g.kv + g.page_elems(layer, page, kvh, kind);
    const int64_t o = kind == 0 ? key_elem(slot, d, g.head_dim) : (int64_t)d * p.page_size + slot;
    base[o] = src[e];
  }
}

// ctx_lens[i] += n_new[i] (prefill bookkeeping, device side).
__global__ void k_add_ctx(int n, int32_t* ctx, const int32_t* add) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) ctx[i] += add[i];
}

}  // namespace

// ---------------------------------------------------------------- launchers
void launch_pool_init(const PoolDev& p, hipStream_t st) {
  k_pool_init<<<1024, 256, 0, st>>>(p);
}
void launch_grow(const PoolDev& p, int n, const int32_t* seq, const int32_t* a, const int32_t* b,
                 int mode, hipStream_t st) {
  k_grow<<<1, kBT, 0, st>>>(p, n, seq, a, b, mode);
}
void launch_verify_setup(const PoolDev& p, const VerifySetupArgs& a, const StepMeta& m,
                         hipStream_t st) {
  k_verify_setup<<<1, kBT, 0, st>>>(p, a, m);
}
void launch_commit(const PoolDev& p, int B, const int32_t* seq, int32_t* ctx, const int32_t* acc,
                   uint32_t commit_seq, hipStream_t st) {
  k_commit<<<1, kBT, 0, st>>>(p, B, seq, ctx, acc, commit_seq);
}
void launch_free(const PoolDev& p, int n, const int32_t* seq, hipStream_t st) {
  k_free<<<1, kBT, 0, st>>>(p, n, seq);
}
void launch_fork(const PoolDev& p, int src, int dst, int npg, hipStream_t st) {
  k_fork<<<1, 1024, 0, st>>>(p, src, dst, npg);
}
void launch_kv_load(const PoolDev& p, const KvGeom& g, int seq, int layer, int pos0, int n,
                    const bf16_t* src, hipStream_t st) {
  const int64_t total = (int64_t)2 * g.n_kv_heads * n * g.head_dim;
  const int blocks = (int)std::min<int64_t>((total + 255) / 256, 65536);
  k_kv_load<<<blocks, 256, 0, st>>>(p, g, seq, layer, pos0, n, src);
}
void launch_add_ctx(int n, int32_t* ctx, const int32_t* add, hipStream_t st) {
  k_add_ctx<<<cdiv_i(n, 256), 256, 0, st>>>(n, ctx, add);
}
