// Kernel arguments of the lm-head log-prob operations, built from a plan and
// the caller's pointers.  The C ABI entry points launch with exactly these
// arguments, and the host bounds replay (bounds.cpp) replays the same ones.
#pragma once

#include "kernels.h"
#include "plan.h"

namespace rlk {

inline LogprobArgs logprob_args(const LogprobPlan &plan, const void *hidden_states, const void *w_lm,
                                const int32_t *target, float inv_temperature, float *logprob, float *lse,
                                unsigned char *ws) {
    LogprobArgs a{};
    a.hidden = static_cast<const uint16_t *>(hidden_states);
    a.w = static_cast<const uint16_t *>(w_lm);
    a.target = target;
    a.logprob = logprob;
    a.lse = lse;
    a.pm = reinterpret_cast<float *>(ws + plan.off_m);
    a.pl = reinterpret_cast<float *>(ws + plan.off_l);
    a.zt = reinterpret_cast<float *>(ws + plan.off_zt);
    a.R = plan.R;
    a.H = plan.H;
    a.V = plan.V;
    a.n_vocab_tiles = static_cast<int32_t>(plan.n_vocab_tiles);
    a.n_row_tiles = static_cast<int32_t>(plan.n_row_tiles);
    a.inv_temperature = inv_temperature;
    a.dp_tiles = plan.n_dp_tiles;
    a.tail_tiles = plan.n_tail_tiles;
    a.splits = plan.tail_splits;
    a.part = reinterpret_cast<float *>(ws + plan.off_part);
    a.narrow_v0 = plan.narrow_v0;
    a.narrow_tiles = plan.narrow_tiles;
    a.narrow_slot0 = plan.narrow_slot0;
    a.narrow_tm = plan.narrow_tm;
    a.n_partials = plan.n_partials;
    return a;
}

// The launches of the backward's chunk starting at row c0: the probability
// pass (f: whole tiles, then, with a tail split, the tail tiles' parts and
// their reduce), then the vocabulary GEMM and the finish kernel (b).
inline void logprob_bwd_chunk_args(const LogprobBwdPlan &plan, int64_t c0, const uint16_t *hid, const uint16_t *w,
                                   const int32_t *target, float inv_temperature, const float *lse,
                                   const float *grad_logprob, float *grad_hidden, unsigned char *ws, LogprobArgs *f,
                                   LogprobBwdArgs *b) {
    const int64_t n = std::min(plan.chunk_rows, plan.R - c0);
    const int32_t row_tiles = static_cast<int32_t>((n + kRowTile - 1) / kRowTile);
    uint16_t *probs = reinterpret_cast<uint16_t *>(ws + plan.off_probs);
    *f = LogprobArgs{};
    f->hidden = hid + c0 * plan.H;
    f->w = w;
    f->target = target + c0;
    f->R = n;
    f->H = plan.H;
    f->V = plan.V;
    f->n_vocab_tiles = static_cast<int32_t>(plan.n_vocab_tiles);
    f->n_row_tiles = row_tiles;
    f->inv_temperature = inv_temperature;
    f->lse_in = lse + c0;
    f->probs = probs;
    const TailSplit ts = bwd_probs_tail(plan, n);
    f->dp_tiles = ts.dp_tiles;
    f->tail_tiles = ts.tail_tiles;
    f->splits = ts.splits;
    f->part = reinterpret_cast<float *>(ws + plan.off_part);
    *b = LogprobBwdArgs{};
    b->w = w;
    b->target = target + c0;
    b->grad = grad_logprob + c0;
    b->dh = grad_hidden + c0 * plan.H;
    b->probs = probs;
    b->dpart = plan.splits > 1 ? reinterpret_cast<float *>(ws + plan.off_part) : b->dh;
    b->rows = n;
    b->H = plan.H;
    b->V = plan.V;
    b->n_vsteps = plan.n_vsteps;
    b->n_row_tiles = row_tiles;
    b->n_h_tiles = plan.n_h_tiles;
    b->splits = plan.splits;
    b->steps_per_split = plan.steps_per_split;
    b->inv_temperature = inv_temperature;
}

// The two launches of the sampling head's chunk starting at row c0: the
// logits tile kernels (f: whole tiles, then the last round's narrow tiles if
// any) and the selection kernel (s).
inline void sample_chunk_args(const SamplePlan &plan, int64_t c0, const uint16_t *hid, const uint16_t *w,
                              const float *inv_temperature, float top_p, const float *uniform, int32_t *token,
                              float *logprob, unsigned char *ws, LogprobArgs *f, SampleArgs *s) {
    const int64_t n = std::min(plan.chunk_rows, plan.R - c0);
    float *logits = reinterpret_cast<float *>(ws + plan.off_logits);
    float *pm = reinterpret_cast<float *>(ws + plan.off_pm);
    *f = LogprobArgs{};
    f->hidden = hid + c0 * plan.H;
    f->w = w;
    f->R = n;
    f->H = plan.H;
    f->V = plan.V;
    f->n_vocab_tiles = static_cast<int32_t>(plan.n_vocab_tiles);
    f->n_row_tiles = static_cast<int32_t>((n + kRowTile - 1) / kRowTile);
    f->inv_temperature = 1.f;
    f->inv_t_rows = inv_temperature + c0;
    f->logits = logits;
    f->ld = plan.ld;
    f->pm = pm;
    const TileRounds tr = plan_tile_rounds(n, plan.V);
    f->dp_tiles = tr.dp_tiles;
    f->narrow_v0 = tr.narrow_v0;
    f->narrow_tiles = tr.narrow_tiles;
    f->narrow_slot0 = tr.narrow_slot0;
    f->narrow_tm = tr.narrow_tm;
    f->n_partials = tr.n_partials;
    *s = SampleArgs{};
    s->logits = logits;
    s->pm = pm;
    s->uniform = uniform + c0;
    s->token = token + c0;
    s->logprob = logprob ? logprob + c0 : nullptr;
    s->rows = n;
    s->ld = plan.ld;
    s->V = plan.V;
    s->n_partials = static_cast<int32_t>(tr.n_partials);
    s->top_p = top_p;
}

}  // namespace rlk
