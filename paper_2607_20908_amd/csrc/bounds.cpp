// Host replay of the global memory accesses of the lm-head log-prob kernels
// (rl_token_logprob and rl_token_logprob_backward), for tests: every launch
// of a call is replayed workgroup by workgroup and lane by lane with the
// arguments the entry point builds (logprob_args.h) and the index arithmetic
// the kernels use (tile_index.h), and every load and store is checked to lie
// inside the allocation, or workspace section, it must fall in.  Allocations
// get disjoint fake base addresses; nothing touches device memory.
//
// Staged loads: a workgroup loads stage min(slot, nks - 1) for every slot it
// issues, and each address is affine and non-decreasing in that clamped stage
// index, so the first and last stage bound every stage's access; with
// every_stage set, every issued slot is replayed instead.  Data-dependent
// accesses (the target's weight row in the finish kernel, the target logit's
// store) are checked at both ends of the range the kernel's guard admits.
#include <algorithm>
#include <atomic>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "decode_args.h"
#include "decode_index.h"
#include "extend_args.h"
#include "extend_index.h"
#include "kernels.h"
#include "logprob_args.h"
#include "plan.h"
#include "rl_kernels.h"
#include "tile_index.h"

namespace rlk {
namespace {

struct Region {
    const char *name;
    uint64_t base, size;   // fake address and bytes
};

class Replay {
  public:
    // shrink: index of the region (in the order added) to make 16 bytes
    // smaller than the entry point requires, or -1
    Replay(bool every_stage, int shrink) : every_stage_(every_stage), shrink_(shrink) {}

    int add(const char *name, uint64_t size) {
        const uint64_t base = static_cast<uint64_t>(regions_.size() + 1) << 44;
        return push({name, base, size});
    }
    // a section [off, off + size) of region `parent`, checked on its own
    int section(const char *name, int parent, uint64_t off, uint64_t size) {
        return push({name, regions_[parent].base + off, size});
    }
    int regions() const { return static_cast<int>(regions_.size()); }
    uint64_t base(int r) const { return regions_[r].base; }
    template <class T>
    T *ptr(int r) const {
        return reinterpret_cast<T *>(static_cast<uintptr_t>(regions_[r].base));
    }
    static uint64_t addr(const void *p) { return static_cast<uint64_t>(reinterpret_cast<uintptr_t>(p)); }
    bool every_stage() const { return every_stage_; }

    // Replays blocks [0, blocks) of one launch on the host's cores.
    template <class F>
    void launch(const char *kernel, int64_t blocks, F body) {
        ++launches_;
        const int nt = static_cast<int>(std::max<unsigned>(1u, std::min<unsigned>(8u, std::thread::hardware_concurrency())));
        std::atomic<int64_t> next{0};
        auto work = [&]() {
            Lane ln{this, kernel, 0, 0, 0, 0};
            for (;;) {
                const int64_t b0 = next.fetch_add(64);
                if (b0 >= blocks) break;
                for (int64_t b = b0; b < std::min(blocks, b0 + 64); ++b) {
                    ln.block = b;
                    body(b, ln);
                }
            }
            accesses_ += ln.n;
            violations_ += ln.bad;
        };
        std::vector<std::thread> ts;
        for (int i = 1; i < nt; ++i) ts.emplace_back(work);
        work();
        for (auto &t : ts) t.join();
    }

    // Per-host-thread checker of one launch.
    struct Lane {
        Replay *rp;
        const char *kernel;
        int64_t block;
        int thread;
        uint64_t n, bad;
        void check(int region, uint64_t a, uint64_t bytes, const char *what) {
            ++n;
            const Region &r = rp->regions_[region];
            if (a >= r.base && bytes <= r.size && a - r.base <= r.size - bytes) return;
            ++bad;
            rp->note(kernel, block, thread, what, r, a, bytes);
        }
    };

    void report(rl_bounds_report *rep) const {
        rep->accesses = accesses_;
        rep->violations = violations_;
        rep->launches = launches_;
        rep->regions = static_cast<int32_t>(regions_.size());
        std::snprintf(rep->first_violation, sizeof(rep->first_violation), "%s", first_.c_str());
    }

  private:
    int push(Region r) {
        if (static_cast<int>(regions_.size()) == shrink_) r.size = r.size >= 16 ? r.size - 16 : 0;
        regions_.push_back(r);
        return static_cast<int>(regions_.size()) - 1;
    }
    void note(const char *kernel, int64_t block, int thread, const char *what, const Region &r, uint64_t a,
              uint64_t bytes) {
        std::lock_guard<std::mutex> g(mu_);
        if (!first_.empty()) return;
        char buf[256];
        std::snprintf(buf, sizeof(buf), "%s block %lld thread %d: %s of %llu bytes at offset %lld of %s (%llu bytes)",
                      kernel, static_cast<long long>(block), thread, what, static_cast<unsigned long long>(bytes),
                      static_cast<long long>(a - r.base), r.name, static_cast<unsigned long long>(r.size));
        first_ = buf;
    }

    bool every_stage_;
    int shrink_;
    std::vector<Region> regions_;
    std::atomic<uint64_t> accesses_{0}, violations_{0};
    int launches_ = 0;
    std::mutex mu_;
    std::string first_;
};

// The stage slots a workgroup issues for one operand: slots 0 .. last_slot
// (each loading stage min(slot, nks - 1)), or the two that load the first and
// the last stage.
std::vector<int> stage_slots(const Replay &rp, int nks, int last_slot) {
    std::vector<int> s;
    if (rp.every_stage()) {
        for (int i = 0; i <= last_slot; ++i) s.push_back(i);
    } else {
        s.push_back(0);
        if (nks - 1 > 0) s.push_back(nks - 1);
    }
    return s;
}

struct TileRegions {
    int hidden, w, target, pm, pl, zt, part, lse_in, probs, inv_t, logits;
};

// logprob_tile_kernel<WS, MODE, TM> over `blocks` workgroups of kTileWaves
// wave64s.
void replay_tile(Replay &rp, const char *name, int mode, int TM, int WS, const LogprobArgs &a, int64_t blocks,
                 const TileRegions &rg) {
    rp.launch(name, blocks, [&](int64_t b, Replay::Lane &ln) {
        const TileCoord tc = tile_coord(mode, TM, b, a);
        const int VW = 64 * TM, WBLK = VW / 64, HBLK = 32 / kTileWaves;   // 1 KB blocks per wave per stage
        const int64_t H = a.H, r0 = tc.rt * kRowTile;
        const int wlast = stage_last(VW, a.V, tc.v0), hlast = stage_last(kRowTile, a.R, r0);
        ln.thread = 0;
        if (tc.nks < 1 || wlast < 0 || hlast < 0) {
            ln.check(rg.w, 0, 1, "tile with no hidden step, vocab entry or row");
            return;
        }
        const uint64_t wg = Replay::addr(a.w) + static_cast<uint64_t>(tc.v0 * H) * 2;
        const uint64_t hg = Replay::addr(a.hidden) + static_cast<uint64_t>(r0 * H) * 2;
        // the hidden rows of slots 0 .. nks - 1 + HS, the weights of 0 .. nks - 1 + WS
        const std::vector<int> hs = stage_slots(rp, tc.nks, tc.nks - 1 + tile_hidden_stages(TM)),
                               ws = stage_slots(rp, tc.nks, tc.nks - 1 + WS);
        for (int wave = 0; wave < kTileWaves; ++wave)
            for (int lane = 0; lane < 64; ++lane) {
                ln.thread = wave * 64 + lane;
                for (int j = 0; j < WBLK; ++j) {
                    const int row = stage_row(wave * WBLK + j, lane);
                    const uint32_t voff = stage_voff(row, wlast, H, stage_chunk(row, lane));
                    for (int slot : ws) ln.check(rg.w, wg + stage_k0(tc.kb, slot, tc.nks) * 2 + voff, 16, "weight stage load");
                }
                for (int j = 0; j < HBLK; ++j) {
                    const int row = stage_row(wave * HBLK + j, lane);
                    const uint32_t voff = stage_voff(row, hlast, H, stage_chunk(row, lane));
                    for (int slot : hs) ln.check(rg.hidden, hg + stage_k0(tc.kb, slot, tc.nks) * 2 + voff, 16, "hidden stage load");
                }
            }
        // epilogues
        const uint64_t tgt = Replay::addr(a.target);
        for (int wave = 0; wave < kTileWaves; ++wave) {
            const int wm = wave & 1, wn = wave >> 1;   // vocab half, 64-row quarter
            for (int lane = 0; lane < 64; ++lane) {
                ln.thread = wave * 64 + lane;
                const int l32 = lane & 31, h2 = lane >> 5;
                if (mode == kLogits) {
                    // the tempered logits of the wave's 32 TM vocab entries
                    const int64_t vbase = tc.v0 + wm * 32 * TM;
                    for (int tn = 0; tn < 2; ++tn) {
                        const int64_t rr = r0 + wn * 64 + tn * 32 + l32;
                        if (rr >= a.R) continue;
                        ln.check(rg.inv_t, Replay::addr(a.inv_t_rows) + rr * 4, 4, "inverse temperature load");
                        for (int tm = 0; tm < TM; ++tm)
                            for (int q = 0; q < 4; ++q)
                                ln.check(rg.logits,
                                         Replay::addr(a.logits) + (rr * a.ld + vbase + 4 * h2 + tm * 32 + 8 * q) * 4,
                                         16, "logits store");
                    }
                    continue;
                }
                if (mode == kPartialK) {
                    for (int tm = 0; tm < 4; ++tm)
                        for (int tn = 0; tn < 2; ++tn)
                            for (int q = 0; q < 4; ++q)
                                ln.check(rg.part, Replay::addr(a.part) + part_elem(b, wm, wn * 2 + tn, tm, q, lane) * 4,
                                         16, "tail part store");
                    continue;
                }
                for (int tn = 0; tn < 2; ++tn) {
                    const int row = wn * 64 + tn * 32 + l32;
                    const int64_t rr = r0 + row;
                    if (mode == kBwdProbs) {
                        if (rr < a.R) {
                            ln.check(rg.target, tgt + rr * 4, 4, "target load");
                            ln.check(rg.lse_in, Replay::addr(a.lse_in) + rr * 4, 4, "lse load");
                        }
                        const uint64_t pb = Replay::addr(a.probs) +
                                            probs_block(tc.rt, a.n_vocab_tiles * 4LL, tc.vt * 4 + wm * 2) * 2;
                        for (int tm = 0; tm < 4; ++tm)
                            for (int q = 0; q < 4; ++q)
                                ln.check(rg.probs, pb + probs_store_off(tm, q, row, h2) * 2, 8, "probability store");
                    } else if (rr < a.R) {   // forward: the row's target, and its logit if the tile holds it
                        ln.check(rg.target, tgt + rr * 4, 4, "target load");
                        ln.check(rg.zt, Replay::addr(a.zt) + rr * 4, 4, "target logit store");
                    }
                }
            }
        }
        if (mode == kLogits)
            for (int tid = 0; tid < 256; ++tid) {
                ln.thread = tid;
                const int64_t rr = r0 + tid;
                if (rr < a.R) ln.check(rg.pm, Replay::addr(a.pm) + (tc.vt * a.R + rr) * 4, 4, "row maximum store");
            }
        if (mode == kFwd || mode == kNarrow)
            for (int tid = 0; tid < 256; ++tid) {
                ln.thread = tid;
                const int64_t rr = r0 + tid;
                if (rr < a.R) {
                    ln.check(rg.pm, Replay::addr(a.pm) + (tc.vt * a.R + rr) * 4, 4, "partial max store");
                    ln.check(rg.pl, Replay::addr(a.pl) + (tc.vt * a.R + rr) * 4, 4, "partial sum store");
                }
            }
    });
}

// logprob_tail_reduce_kernel: 8 workgroups of 128 threads per tail tile.
void replay_tail_reduce(Replay &rp, const LogprobArgs &t, const TileRegions &rg) {
    rp.launch("logprob_tail_reduce_kernel", t.tail_tiles * 8, [&](int64_t b, Replay::Lane &ln) {
        const int64_t j = b >> 3;
        const int rb = static_cast<int>(b & 7);
        int64_t vt, rt;
        tile_of_logical(t.tile_base + j, t.n_vocab_tiles, t.n_row_tiles, &vt, &rt);
        for (int tid = 0; tid < 128; ++tid) {
            ln.thread = tid;
            const int wm = tid >> 6, lane = tid & 63, l32 = lane & 31;
            for (int sp = 0; sp < t.splits; ++sp)
                for (int tm = 0; tm < 4; ++tm)
                    for (int q = 0; q < 4; ++q)
                        ln.check(rg.part, Replay::addr(t.part) + part_elem(j * t.splits + sp, wm, rb, tm, q, lane) * 4,
                                 16, "tail part load");
            const int64_t rr = rt * kRowTile + rb * 32 + l32;
            if (rr < t.R) {
                ln.check(rg.target, Replay::addr(t.target) + rr * 4, 4, "target load");
                ln.check(rg.zt, Replay::addr(t.zt) + rr * 4, 4, "target logit store");
            }
            if (tid < 32) {
                const int64_t r = rt * kRowTile + rb * 32 + tid;
                if (r < t.R) {
                    ln.check(rg.pm, Replay::addr(t.pm) + (vt * t.R + r) * 4, 4, "partial max store");
                    ln.check(rg.pl, Replay::addr(t.pl) + (vt * t.R + r) * 4, 4, "partial sum store");
                }
            }
        }
    });
}

// logprob_probs_tail_reduce_kernel: 8 workgroups of 128 threads per tail
// tile of the backward's probability pass.
void replay_probs_tail_reduce(Replay &rp, const LogprobArgs &t, const TileRegions &rg) {
    rp.launch("logprob_probs_tail_reduce_kernel", t.tail_tiles * 8, [&](int64_t b, Replay::Lane &ln) {
        const int64_t j = b >> 3;
        const int rb = static_cast<int>(b & 7);
        int64_t vt, rt;
        tile_of_logical(t.tile_base + j, t.n_vocab_tiles, t.n_row_tiles, &vt, &rt);
        for (int tid = 0; tid < 128; ++tid) {
            ln.thread = tid;
            const int wm = tid >> 6, lane = tid & 63, l32 = lane & 31, h2 = lane >> 5;
            for (int sp = 0; sp < t.splits; ++sp)
                for (int tm = 0; tm < 4; ++tm)
                    for (int q = 0; q < 4; ++q)
                        ln.check(rg.part, Replay::addr(t.part) + part_elem(j * t.splits + sp, wm, rb, tm, q, lane) * 4,
                                 16, "tail part load");
            const int row = rb * 32 + l32;
            const int64_t rr = rt * kRowTile + row;
            if (rr < t.R) {
                ln.check(rg.target, Replay::addr(t.target) + rr * 4, 4, "target load");
                ln.check(rg.lse_in, Replay::addr(t.lse_in) + rr * 4, 4, "lse load");
            }
            const uint64_t pb = Replay::addr(t.probs) + probs_block(rt, t.n_vocab_tiles * 4LL, vt * 4 + wm * 2) * 2;
            for (int tm = 0; tm < 4; ++tm)
                for (int q = 0; q < 4; ++q)
                    ln.check(rg.probs, pb + probs_store_off(tm, q, row, h2) * 2, 8, "probability store");
        }
    });
}

// sample_top_p_kernel: one workgroup per row.  Its reads of the row's logits
// go to float4 groups below (V + 3) / 4 and to the drawn id (< V); which ones
// depends on the data, so the replay checks the whole range the kernel may
// touch: every group of the row, the row maxima of every partial slot, and
// the per-row input and outputs.
void replay_select(Replay &rp, const SampleArgs &s, int pm_r, int logits_r, int u_r, int tok_r, int lp_r) {
    rp.launch("sample_top_p_kernel", s.rows, [&](int64_t r, Replay::Lane &ln) {
        ln.thread = 0;
        const int64_t nvec = (s.V + 3) / 4;
        const uint64_t y = Replay::addr(s.logits) + static_cast<uint64_t>(r * s.ld) * 4;
        for (int64_t g = 0; g < nvec; ++g) ln.check(logits_r, y + g * 16, 16, "logits load");
        for (int64_t t = 0; t < s.n_partials; ++t)
            ln.check(pm_r, Replay::addr(s.pm) + (t * s.rows + r) * 4, 4, "row maximum load");
        ln.check(u_r, Replay::addr(s.uniform) + r * 4, 4, "uniform load");
        ln.check(tok_r, Replay::addr(s.token) + r * 4, 4, "token store");
        if (s.logprob) ln.check(lp_r, Replay::addr(s.logprob) + r * 4, 4, "log-prob store");
    });
}

// The combine kernel launch_logprob picks for a.R rows.
void replay_combine(Replay &rp, const LogprobArgs &a, const TileRegions &rg, int logprob_r, int lse_r) {
    const int kind = logprob_combine_kind(a.R);
    const int64_t blocks = kind == kCombineBlock ? a.R : kind == kCombineWave ? (a.R + 3) / 4 : (a.R + 255) / 256;
    rp.launch(kind == kCombineBlock ? "logprob_combine_block_kernel"
                                    : kind == kCombineWave ? "logprob_combine_wave_kernel" : "logprob_combine_row_kernel",
              blocks, [&](int64_t b, Replay::Lane &ln) {
                  for (int tid = 0; tid < 256; ++tid) {
                      ln.thread = tid;
                      int64_t r, vt0, step;
                      bool finisher;
                      if (kind == kCombineBlock) {
                          r = b, vt0 = tid, step = 256, finisher = tid == 0;
                      } else if (kind == kCombineWave) {
                          r = b * 4 + (tid >> 6), vt0 = tid & 63, step = 64, finisher = (tid & 63) == 0;
                      } else {
                          r = b * 256 + tid, vt0 = 0, step = 1, finisher = true;
                      }
                      if (r >= a.R) continue;
                      for (int64_t vt = vt0; vt < a.n_partials; vt += step) {
                          ln.check(rg.pm, Replay::addr(a.pm) + (vt * a.R + r) * 4, 4, "partial max load");
                          ln.check(rg.pl, Replay::addr(a.pl) + (vt * a.R + r) * 4, 4, "partial sum load");
                      }
                      if (finisher) {
                          ln.check(rg.target, Replay::addr(a.target) + r * 4, 4, "target load");
                          ln.check(rg.zt, Replay::addr(a.zt) + r * 4, 4, "target logit load");
                          ln.check(logprob_r, Replay::addr(a.logprob) + r * 4, 4, "logprob store");
                          if (a.lse) ln.check(lse_r, Replay::addr(a.lse) + r * 4, 4, "lse store");
                      }
                  }
              });
}

// logprob_bwd_gemm_kernel<WS>.
void replay_bwd_gemm(Replay &rp, const LogprobBwdArgs &a, int probs_r, int w_r, int out_r) {
    const int WS = tile_weight_stages(a.n_row_tiles);
    rp.launch("logprob_bwd_gemm_kernel", bwd_gemm_blocks(a), [&](int64_t b, Replay::Lane &ln) {
        int split, ht, rt;
        gemm_tile_of(b, a.n_h_tiles, a.n_row_tiles, a.splits, &split, &ht, &rt);
        const int H = a.H, h0 = ht * 256;
        const int ks0 = split * a.steps_per_split;
        const int nks = std::min(a.steps_per_split, a.n_vsteps - ks0);
        ln.thread = 0;
        if (nks < 1 || rt >= a.n_row_tiles || h0 >= H) {
            ln.check(out_r, 0, 1, "workgroup outside the vocabulary, rows or hidden size");
            return;
        }
        const int clast = bwd_clast(H, h0);
        const std::vector<int> as = stage_slots(rp, nks, nks + 1), bs = stage_slots(rp, nks, nks - 1 + WS);
        constexpr int BLK = 32 / kBwdGemmWaves;   // 1 KB blocks per wave per operand per stage
        for (int wave = 0; wave < kBwdGemmWaves; ++wave)
            for (int lane = 0; lane < 64; ++lane) {
                ln.thread = wave * 64 + lane;
                for (int j = 0; j < BLK; ++j) {
                    const int blk = wave * BLK + j;
                    for (int slot : as)
                        ln.check(probs_r,
                                 Replay::addr(a.probs) + bwd_a_base(rt, a.n_vsteps, ks0, slot, nks, blk) * 2 +
                                     bwd_a_voff(lane),
                                 16, "probability stage load");
                    const int row = bwd_b_row(blk, lane);
                    const int c = bwd_b_chunk(row, lane);
                    for (int slot : bs) {
                        const int64_t first = bwd_b_first(ks0, slot, nks, blk);
                        const uint64_t base = Replay::addr(a.w) + (bwd_b_base_row(first, a.V) * H + h0) * 2;
                        const uint32_t voff = bwd_b_voff(lane, bwd_b_pair(first, a.V), c, clast, H);
                        ln.check(w_r, base + voff, 16, "weight stage load");
                        // the row the lane must read: its band row, clamped to the vocabulary
                        const int64_t want = std::min<int64_t>(first + (lane >> 5), a.V - 1);
                        if (base + voff != Replay::addr(a.w) + (want * H + h0 + 8 * std::min(c, clast)) * 2)
                            ln.check(w_r, 0, static_cast<uint64_t>(1) << 63, "weight load not at its clamped row");
                    }
                }
            }
        const int64_t rows_pad = static_cast<int64_t>(a.n_row_tiles) * 256;
        const uint64_t out = Replay::addr(a.dpart) + bwd_out_base(split, rows_pad, rt, H, h0) * 4;
        const int64_t rlim = a.rows - static_cast<int64_t>(rt) * 256;
        for (int wave = 0; wave < kBwdGemmWaves; ++wave) {
            const int wm = wave & 1, wn = wave >> 1;   // row half, hidden quarter
            for (int lane = 0; lane < 64; ++lane) {
                ln.thread = wave * 64 + lane;
                const int l32 = lane & 31, h2 = lane >> 5;
                for (int tn = 0; tn < 2; ++tn) {
                    const int h = wn * 64 + tn * 32 + l32;
                    if (h0 + h >= H) continue;
                    for (int tm = 0; tm < 4; ++tm)
                        for (int i = 0; i < 16; ++i) {
                            const int row = wm * 128 + tm * 32 + 8 * (i >> 2) + 4 * h2 + (i & 3);
                            if (row < rlim) ln.check(out_r, out + bwd_out_off(row, H, h) * 4, 4, "partial sum store");
                        }
                }
            }
        }
    });
}

// logprob_bwd_finish_kernel: one thread per 4 hidden entries of a row.
void replay_bwd_finish(Replay &rp, const LogprobBwdArgs &a, int part_r, int w_r, int target_r, int grad_r, int dh_r) {
    const int64_t per_row = a.H / 4;
    rp.launch("logprob_bwd_finish_kernel", bwd_finish_blocks(a), [&](int64_t b, Replay::Lane &ln) {
        const int64_t rows_pad = static_cast<int64_t>(a.n_row_tiles) * 256;
        for (int tid = 0; tid < kBwdFinishThreads; ++tid) {
            ln.thread = tid;
            const int64_t idx = b * kBwdFinishThreads + tid;
            if (idx >= a.rows * per_row) continue;
            const int64_t r = idx / per_row;
            const int h = static_cast<int>(idx % per_row) * 4;
            ln.check(target_r, Replay::addr(a.target) + r * 4, 4, "target load");
            // a valid target t in [0, V): the split sums, W[t] and the gradient
            for (int sp = 0; sp < a.splits; ++sp)
                ln.check(part_r, Replay::addr(a.dpart) + bwd_part_elem(sp, rows_pad, r, a.H, h) * 4, 16,
                         "partial sum load");
            for (int64_t t : {static_cast<int64_t>(0), static_cast<int64_t>(a.V - 1)})
                ln.check(w_r, Replay::addr(a.w) + (t * a.H + h) * 2, 8, "target weight load");
            ln.check(grad_r, Replay::addr(a.grad) + r * 4, 4, "gradient load");
            ln.check(dh_r, Replay::addr(a.dh) + (r * a.H + h) * 4, 16, "gradient store");
        }
    });
}

}  // namespace
}  // namespace rlk

extern "C" rl_status rl_debug_logprob_bounds(int32_t op, int64_t rows, int32_t hidden, int32_t vocab,
                                             int32_t every_stage, int32_t shrink_region, rl_bounds_report *report) {
    using namespace rlk;
    if (!report) return RL_ERR_NULL_POINTER;
    std::memset(report, 0, sizeof(*report));
    std::string err;
    Replay rp(every_stage != 0, shrink_region);
    if (op == 0) {
        LogprobPlan plan;
        const rl_status st = plan_logprob(rows, hidden, vocab, &plan, &err);
        if (st != RL_OK) return st;
        if (rows == 0) return RL_OK;
        TileRegions rg{};
        rg.hidden = rp.add("hidden", static_cast<uint64_t>(rows) * hidden * 2);
        rg.w = rp.add("w_lm", static_cast<uint64_t>(vocab) * hidden * 2);
        rg.target = rp.add("target", static_cast<uint64_t>(rows) * 4);
        const int lp = rp.add("logprob", static_cast<uint64_t>(rows) * 4);
        const int ls = rp.add("lse", static_cast<uint64_t>(rows) * 4);
        const int ws = rp.add("workspace", plan.total_bytes);
        rg.pm = rp.section("workspace partial max", ws, plan.off_m, static_cast<uint64_t>(plan.n_partials) * rows * 4);
        rg.pl = rp.section("workspace partial sum", ws, plan.off_l, static_cast<uint64_t>(plan.n_partials) * rows * 4);
        rg.zt = rp.section("workspace target logits", ws, plan.off_zt, static_cast<uint64_t>(rows) * 4);
        rg.part = rp.section("workspace tail parts", ws, plan.off_part, plan.total_bytes - plan.off_part);
        const LogprobArgs a = logprob_args(plan, rp.ptr<void>(rg.hidden), rp.ptr<void>(rg.w), rp.ptr<int32_t>(rg.target),
                                           1.f, rp.ptr<float>(lp), rp.ptr<float>(ls), rp.ptr<unsigned char>(ws));
        // the launches of launch_logprob, in order
        LogprobArgs d = a;
        d.tile_base = 0;
        d.tile_count = a.dp_tiles;
        replay_tile(rp, "logprob_tile_kernel<kFwd>", kFwd, 4, tile_weight_stages(a.n_row_tiles), d, d.tile_count, rg);
        if (a.narrow_tiles > 0)
            replay_tile(rp, "logprob_tile_kernel<kNarrow>", kNarrow, a.narrow_tm, 3, a, a.narrow_tiles * a.n_row_tiles,
                        rg);
        if (a.tail_tiles > 0) {
            LogprobArgs t = a;
            t.tile_base = a.dp_tiles;
            t.tile_count = a.tail_tiles;
            replay_tile(rp, "logprob_tile_kernel<kPartialK>", kPartialK, 4, tile_weight_stages(a.n_row_tiles), t,
                        a.tail_tiles * a.splits, rg);
            replay_tail_reduce(rp, t, rg);
        }
        replay_combine(rp, a, rg, lp, ls);
    } else if (op == 1) {
        LogprobBwdPlan plan;
        const rl_status st = plan_logprob_bwd(rows, hidden, vocab, &plan, &err);
        if (st != RL_OK) return st;
        if (rows == 0) return RL_OK;
        TileRegions rg{};
        rg.hidden = rp.add("hidden", static_cast<uint64_t>(rows) * hidden * 2);
        rg.w = rp.add("w_lm", static_cast<uint64_t>(vocab) * hidden * 2);
        rg.target = rp.add("target", static_cast<uint64_t>(rows) * 4);
        rg.lse_in = rp.add("lse", static_cast<uint64_t>(rows) * 4);
        const int grad = rp.add("grad_logprob", static_cast<uint64_t>(rows) * 4);
        const int dh = rp.add("grad_hidden", static_cast<uint64_t>(rows) * hidden * 4);
        const int ws = rp.add("workspace", plan.total_bytes);
        const uint64_t rows_pad = static_cast<uint64_t>(plan.chunk_row_tiles) * kRowTile;
        rg.probs = rp.section("workspace probabilities", ws, plan.off_probs,
                              rows_pad * static_cast<uint64_t>(plan.n_vsteps) * kHiddenStep * 2);
        // one section for the probability tail's parts and the GEMM's split
        // sums (used one after the other within a chunk)
        const bool has_part = plan.total_bytes > plan.off_part;
        const int part = has_part ? rp.section("workspace tail parts and split sums", ws, plan.off_part,
                                               plan.total_bytes - plan.off_part)
                                  : -1;
        rg.part = part;
        const int gemm_out = plan.splits > 1 ? part : dh;
        for (int64_t c0 = 0; c0 < rows; c0 += plan.chunk_rows) {
            LogprobArgs f;
            LogprobBwdArgs b;
            logprob_bwd_chunk_args(plan, c0, rp.ptr<uint16_t>(rg.hidden), rp.ptr<uint16_t>(rg.w),
                                   rp.ptr<int32_t>(rg.target), 1.f, rp.ptr<float>(rg.lse_in), rp.ptr<float>(grad),
                                   rp.ptr<float>(dh), rp.ptr<unsigned char>(ws), &f, &b);
            // the launches of launch_logprob_probs, in order
            LogprobArgs d = f;
            d.tile_base = 0;
            d.tile_count = f.dp_tiles;
            replay_tile(rp, "logprob_tile_kernel<kBwdProbs>", kBwdProbs, 4, tile_weight_stages(f.n_row_tiles), d,
                        d.tile_count, rg);
            if (f.tail_tiles > 0) {
                LogprobArgs t = f;
                t.tile_base = f.dp_tiles;
                t.tile_count = f.tail_tiles;
                replay_tile(rp, "logprob_tile_kernel<kPartialK>", kPartialK, 4, tile_weight_stages(f.n_row_tiles), t,
                            f.tail_tiles * f.splits, rg);
                replay_probs_tail_reduce(rp, t, rg);
            }
            replay_bwd_gemm(rp, b, rg.probs, rg.w, gemm_out);
            replay_bwd_finish(rp, b, gemm_out, rg.w, rg.target, grad, dh);
        }
    } else if (op == 2) {
        SamplePlan plan;
        const rl_status st = plan_sample(rows, hidden, vocab, &plan, &err);
        if (st != RL_OK) return st;
        if (rows == 0) return RL_OK;
        TileRegions rg{};
        rg.hidden = rp.add("hidden", static_cast<uint64_t>(rows) * hidden * 2);
        rg.w = rp.add("w_lm", static_cast<uint64_t>(vocab) * hidden * 2);
        rg.inv_t = rp.add("inv_temperature", static_cast<uint64_t>(rows) * 4);
        const int u = rp.add("uniform", static_cast<uint64_t>(rows) * 4);
        const int tok = rp.add("token", static_cast<uint64_t>(rows) * 4);
        const int lp = rp.add("logprob", static_cast<uint64_t>(rows) * 4);
        const int ws = rp.add("workspace", plan.total_bytes);
        const uint64_t rows_pad = static_cast<uint64_t>((plan.chunk_rows + kRowTile - 1) / kRowTile) * kRowTile;
        rg.logits = rp.section("workspace logits", ws, plan.off_logits, rows_pad * plan.ld * 4);
        rg.pm = rp.section("workspace row maxima", ws, plan.off_pm, static_cast<uint64_t>(plan.pm_slots) * plan.chunk_rows * 4);
        for (int64_t c0 = 0; c0 < rows; c0 += plan.chunk_rows) {
            LogprobArgs f;
            SampleArgs s;
            sample_chunk_args(plan, c0, rp.ptr<uint16_t>(rg.hidden), rp.ptr<uint16_t>(rg.w), rp.ptr<float>(rg.inv_t),
                              0.9f, rp.ptr<float>(u), rp.ptr<int32_t>(tok), rp.ptr<float>(lp),
                              rp.ptr<unsigned char>(ws), &f, &s);
            // the launches of launch_logits and launch_sample_top_p, in order
            LogprobArgs d = f;
            d.tile_base = 0;
            d.tile_count = f.dp_tiles;
            if (d.tile_count > 0)
                replay_tile(rp, "logprob_tile_kernel<kLogits>", kLogits, 4, tile_weight_stages(f.n_row_tiles), d,
                            d.tile_count, rg);
            if (f.narrow_tiles > 0)
                replay_tile(rp, "logprob_tile_kernel<kLogits, narrow>", kLogits, f.narrow_tm, 3, f,
                            f.narrow_tiles * f.n_row_tiles, rg);
            replay_select(rp, s, rg.pm, rg.logits, u, tok, lp);
        }
    } else {
        return RL_ERR_INVALID_SHAPE;
    }
    rp.report(report);
    return RL_OK;
}

// Host replay of rl_extend_attn's global accesses (see the header).
extern "C" rl_status rl_debug_extend_bounds(const rl_decode_shape *shape, const rl_extend_lens *lens,
                                            int32_t every_stage, int32_t shrink_region, rl_bounds_report *report) {
    using namespace rlk;
    if (!report) return RL_ERR_NULL_POINTER;
    std::memset(report, 0, sizeof(*report));
    std::string err;
    ExtendPlan plan;
    const rl_status st = plan_extend(shape, lens, &plan, &err, true);
    if (st != RL_OK) return st;
    if (plan.n_items == 0) return RL_OK;
    Replay rp(every_stage != 0, shrink_region);
    const int64_t D = plan.D, Hq = plan.Hq, Hkv = plan.Hkv;
    const int q_r = rp.add("q", static_cast<uint64_t>(plan.q_rows) * Hq * D * 2);
    const int kp_r = rp.add("k_prefix", static_cast<uint64_t>(plan.prefix_rows) * Hkv * D * 2);
    const int vp_r = rp.add("v_prefix", static_cast<uint64_t>(plan.prefix_rows) * Hkv * D * 2);
    const int ks_r = rp.add("k_suffix", static_cast<uint64_t>(plan.suffix_rows) * Hkv * D * 2);
    const int vs_r = rp.add("v_suffix", static_cast<uint64_t>(plan.suffix_rows) * Hkv * D * 2);
    const int out_r = rp.add("out", static_cast<uint64_t>(plan.q_rows) * Hq * D * 2);
    const int lse_r = rp.add("lse", static_cast<uint64_t>(plan.q_rows) * Hq * 4);
    const int ws_r = rp.add("workspace", plan.total_bytes);
    const int items_r = rp.section("workspace work list", ws_r, 0, static_cast<uint64_t>(plan.n_items) * sizeof(ExtItem));
    rl_decode_ptrs ptrs{};
    ptrs.q = rp.ptr<void>(q_r);
    ptrs.k_prefix = rp.ptr<void>(kp_r);
    ptrs.v_prefix = rp.ptr<void>(vp_r);
    ptrs.k_suffix = rp.ptr<void>(ks_r);
    ptrs.v_suffix = rp.ptr<void>(vs_r);
    ptrs.out = rp.ptr<void>(out_r);
    ptrs.lse = rp.ptr<float>(lse_r);
    const ExtendArgs a = extend_args(plan, ptrs, rp.ptr<void>(ws_r));
    const int lpw = static_cast<int>(kExtTileTokens * D / 512 / kExtWaves);   // 1 KB loads per wave per tile
    const int nkk = static_cast<int>(D / 16), ndt = static_cast<int>(D / 32);
    rp.launch("extend_attn_kernel", plan.n_items, [&](int64_t b, Replay::Lane &ln) {
        const ExtItem &it = plan.items[static_cast<size_t>(b)];
        ln.thread = 0;
        ln.check(items_r, Replay::addr(a.items) + b * sizeof(ExtItem), sizeof(ExtItem), "work item load");
        const ExtGeom g = ext_geom(it, a.r);
        const int64_t stride = ext_tok_stride(a, static_cast<int>(D));
        const int64_t poff = ext_prefix_off(a, it, static_cast<int>(D));
        const int64_t soff = ext_suffix_off(a, it, static_cast<int>(D));
        // tiles replayed: all, or the first and last of the prefix and of the
        // suffix (a lane's address grows with the tile inside a range, and
        // the last tile of a range is the ragged one)
        std::vector<int> tiles;
        if (rp.every_stage()) {
            for (int t = 0; t < g.ntiles; ++t) tiles.push_back(t);
        } else {
            for (int t : {0, g.np - 1, g.np, g.ntiles - 1})
                if (t >= 0 && t < g.ntiles && (tiles.empty() || tiles.back() != t)) tiles.push_back(t);
        }
        for (int wave = 0; wave < kExtWaves; ++wave)
            for (int lane = 0; lane < 64; ++lane) {
                ln.thread = wave * 64 + lane;
                const int l32 = lane & 31, h2 = lane >> 5;
                const int row = wave * kExtRowsPerWave + l32;
                if (row < g.rows) {
                    const int u = it.row_begin + row;
                    const int64_t qrow = ext_q_row(a, it, u);
                    for (int kk = 0; kk < nkk; ++kk)
                        ln.check(q_r, Replay::addr(a.q) + (qrow * D + h2 * 8 + kk * 16) * 2, 16, "query load");
                    for (int dt = 0; dt < ndt; ++dt)
                        for (int q4 = 0; q4 < 4; ++q4)
                            ln.check(out_r, Replay::addr(a.out) + (qrow * D + 4 * h2 + 32 * dt + 8 * q4) * 2, 8,
                                     "output store");
                    if (h2 == 0) ln.check(lse_r, Replay::addr(a.lse) + qrow * 4, 4, "lse store");
                }
                for (int t : tiles) {
                    const bool pre = t < g.np;
                    const int tok0 = ext_tile_tok0(t, g.np), cnt = ext_tile_cnt(t, g.np, it.Lp, g.suf_ctx);
                    const int64_t base = (pre ? poff : soff) + tok0 * stride;
                    const uint64_t kb = Replay::addr(pre ? a.k_prefix : a.k_suffix) + base * 2;
                    const uint64_t vb = Replay::addr(pre ? a.v_prefix : a.v_suffix) + base * 2;
                    for (int j = 0; j < lpw; ++j) {
                        const int e = (wave * lpw + j) * 64 + lane;
                        const int tt = D == 128 ? ext_load_tok<128>(e) : ext_load_tok<64>(e);
                        const int chk = D == 128 ? ext_load_chunk<128>(e) : ext_load_chunk<64>(e);
                        const uint32_t off = cnt == kExtTileTokens ? ext_load_off_full(tt, stride, chk)
                                                                   : ext_load_off(tt, cnt, stride, chk);
                        ln.check(pre ? kp_r : ks_r, kb + off, 16, pre ? "prefix K tile load" : "suffix K tile load");
                        ln.check(pre ? vp_r : vs_r, vb + off, 16, pre ? "prefix V tile load" : "suffix V tile load");
                    }
                }
            }
    });
    rp.report(report);
    return RL_OK;
}

// Host replay of rl_decode_attn's global accesses (see the header).
extern "C" rl_status rl_debug_decode_bounds(const rl_decode_shape *shape, const rl_decode_lens *lens,
                                            int32_t shrink_region, rl_bounds_report *report) {
    using namespace rlk;
    if (!report) return RL_ERR_NULL_POINTER;
    std::memset(report, 0, sizeof(*report));
    std::string err;
    DecodePlan plan;
    const rl_status st = plan_decode(shape, lens, &plan, &err, PlanDetail::kDevice);
    if (st != RL_OK) return st;
    const int64_t S = static_cast<int64_t>(plan.P) * plan.G;
    if (S == 0) return RL_OK;
    Replay rp(false, shrink_region);
    const int64_t D = plan.D, Hq = plan.Hq, Hkv = plan.Hkv;
    const int q_r = rp.add("q", static_cast<uint64_t>(S) * Hq * D * 2);
    const int kp_r = rp.add("k_prefix", static_cast<uint64_t>(plan.prefix_rows) * Hkv * D * 2);
    const int vp_r = rp.add("v_prefix", static_cast<uint64_t>(plan.prefix_rows) * Hkv * D * 2);
    const int ks_r = rp.add("k_suffix", static_cast<uint64_t>(plan.suffix_rows) * Hkv * D * 2);
    const int vs_r = rp.add("v_suffix", static_cast<uint64_t>(plan.suffix_rows) * Hkv * D * 2);
    const int out_r = rp.add("out", static_cast<uint64_t>(S) * Hq * D * 2);
    const int lse_r = rp.add("lse", static_cast<uint64_t>(S) * Hq * 4);
    const int ws_r = rp.add("workspace", plan.total_bytes);
    const int meta_r = rp.section("workspace work list and unit tables", ws_r, 0, plan.meta_bytes);
    const int items_r = rp.section("workspace work list", ws_r, plan.off_items, plan.dev_items.size() * sizeof(DevItem));
    const int pu_r = rp.section("workspace prefix units", ws_r, plan.off_prefix_units, plan.prefix_units.size() * sizeof(DevUnit));
    const int su_r = rp.section("workspace suffix units", ws_r, plan.off_suffix_units, plan.suffix_units.size() * sizeof(DevUnit));
    const uint64_t prow = static_cast<uint64_t>(plan.partial_rows);
    const int pm_r = rp.section("workspace partial max", ws_r, plan.off_m, prow * 4);
    const int pl_r = rp.section("workspace partial sum", ws_r, plan.off_l, prow * 4);
    const int pa_r = rp.section("workspace partial values", ws_r, plan.off_acc, prow * D * 4);
    rl_decode_ptrs ptrs{};
    ptrs.q = rp.ptr<void>(q_r);
    ptrs.k_prefix = rp.ptr<void>(kp_r);
    ptrs.v_prefix = rp.ptr<void>(vp_r);
    ptrs.k_suffix = rp.ptr<void>(ks_r);
    ptrs.v_suffix = rp.ptr<void>(vs_r);
    ptrs.out = rp.ptr<void>(out_r);
    ptrs.lse = rp.ptr<float>(lse_r);
    const DecodeArgs a = decode_args(plan, ptrs, rp.ptr<unsigned char>(ws_r));
    // the work list and unit tables' upload: one copy of meta_bytes (16 bytes
    // per thread) into the start of the workspace
    rp.launch("plan_fetch_kernel", 1, [&](int64_t, Replay::Lane &ln) {
        ln.thread = 0;
        ln.check(meta_r, Replay::addr(a.items), 16, "work list upload (first)");
        ln.check(meta_r, Replay::addr(a.items) + plan.meta_bytes - 16, 16, "work list upload (last)");
    });
    rp.launch("decode_split_kernel", a.n_items, [&](int64_t b, Replay::Lane &ln) {
        const DevItem &it = plan.dev_items[static_cast<size_t>(b)];
        ln.thread = 0;
        ln.check(items_r, Replay::addr(a.items) + b * sizeof(DevItem), sizeof(DevItem), "work item load");
        const int kh = dec_kh(it.meta);
        const bool is_suffix = dec_is_suffix(it.meta);
        const int row_begin = dec_row_begin(it.meta);
        const int rows = dec_item_rows(dec_unit_rows(a, is_suffix), row_begin);
        const int ntok = dec_ntok(it.meta);
        const int64_t stride = dec_tok_stride(a, static_cast<int>(D));
        const int64_t base = dec_kv_base(a, it, DecItem{kh, is_suffix}, static_cast<int>(D));
        const uint64_t kg = Replay::addr(is_suffix ? a.k_suffix : a.k_prefix) + base * 2;
        const uint64_t vg = Replay::addr(is_suffix ? a.v_suffix : a.v_prefix) + base * 2;
        const int kr = is_suffix ? ks_r : kp_r, vr = is_suffix ? vs_r : vp_r;
        // every tile's buffer descriptor lies inside its buffer (the hardware
        // clamps each lane's offset to the descriptor's range); the loads past
        // the last tile have empty ranges
        const int ntiles = (ntok + kTileTokens - 1) / kTileTokens;
        for (int t = 0; t < ntiles; ++t) {
            const int t0 = t * kTileTokens;
            const int64_t first = dec_tile_first(t0, ntok, stride);
            const int range = dec_tile_range(t0, ntok, stride, static_cast<int>(D));
            ln.check(kr, kg + first * 2, static_cast<uint64_t>(range), "K tile descriptor");
            ln.check(vr, vg + first * 2, static_cast<uint64_t>(range), "V tile descriptor");
        }
        // the queries and the partials of the item's rows
        for (int i = 0; i < rows; ++i) {
            ln.thread = i;
            const int64_t qoff = dec_q_off(a, it, DecItem{kh, is_suffix}, row_begin + i, static_cast<int>(D));
            ln.check(q_r, Replay::addr(a.q) + qoff * 2, static_cast<uint64_t>(D) * 2, "query row load");
            const int64_t pr = static_cast<int64_t>(it.partial_row0) + i;
            ln.check(pa_r, Replay::addr(a.pacc) + pr * D * 4, static_cast<uint64_t>(D) * 4, "partial values store");
            ln.check(pm_r, Replay::addr(a.pm) + pr * 4, 4, "partial max store");
            ln.check(pl_r, Replay::addr(a.pl) + pr * 4, 4, "partial sum store");
        }
    });
    const int64_t rows = S * Hq;
    rp.launch("decode_combine_kernel", rows, [&](int64_t idx, Replay::Lane &ln) {
        ln.thread = 0;
        const int64_t s = idx / a.Hq;
        const int h = static_cast<int>(idx % a.Hq);
        const int64_t p = s / a.G;
        const int g = static_cast<int>(s % a.G);
        const int kh = h / a.r, hr = h % a.r;
        ln.check(pu_r, Replay::addr(a.prefix_units) + p * sizeof(DevUnit), sizeof(DevUnit), "prefix unit load");
        ln.check(su_r, Replay::addr(a.suffix_units) + s * sizeof(DevUnit), sizeof(DevUnit), "suffix unit load");
        const DevUnit pu = plan.prefix_units[static_cast<size_t>(p)];
        const DevUnit su = plan.suffix_units[static_cast<size_t>(s)];
        const int64_t Mp = static_cast<int64_t>(a.G) * a.r;
        const int pn = static_cast<int>(pu.nchunks);
        const int n = pn + static_cast<int>(su.nchunks);
        const int64_t pbase = dec_prefix_partial_base(pu, kh, Mp, g, a.r, hr);
        const int64_t sbase = dec_suffix_partial_base(su, kh, a.r, hr);
        for (int j = 0; j < n; ++j) {
            const int64_t pr = dec_partial_row(pbase, sbase, Mp, pn, a.r, j);
            ln.check(pm_r, Replay::addr(a.pm) + pr * 4, 4, "partial max load");
            ln.check(pl_r, Replay::addr(a.pl) + pr * 4, 4, "partial sum load");
            ln.check(pa_r, Replay::addr(a.pacc) + pr * D * 4, static_cast<uint64_t>(D) * 4, "partial values load");
        }
        ln.check(out_r, Replay::addr(a.out) + idx * D * 2, static_cast<uint64_t>(D) * 2, "output row store");
        ln.check(lse_r, Replay::addr(a.lse) + idx * 4, 4, "lse store");
    });
    rp.report(report);
    return RL_OK;
}
