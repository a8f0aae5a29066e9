// State updates of the device-resident decoding loop, shared by the greedy
// head and the sampling variant.  Each runs on one thread after a step's
// tokens are decided; it writes the emitted tokens, the control block of the
// next step (positions, rows, input tokens) and, for self-speculative steps,
// posts the outcome to the host's mailbox.  A self-speculative decision sets
// the next step's rows in ctl->m_next; that step's guard kernel moves them to
// ctl->m if the step the host enqueued is the one decided.
#pragma once

#include "sd_internal.h"

namespace sdk {

__device__ inline void post_mailbox(DevState *st, Mailbox *mb) {
    st->seq += 1;
    __hip_atomic_store(&mb->word, mb_pack(st->seq, st->phase, st->gen_done, st->emitted), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_SYSTEM);
}

// Autoregressive step (Algorithm 1): append tok and feed it back.
__device__ inline void ar_commit(const HeadArgs &h, DevCtl *ctl, int tok) {
    DevState *st = h.st;
    h.out_tokens[st->emitted] = tok;
    st->emitted += 1;
    st->lc += 1;
    st->last = tok;
    ctl->pos += 1;
    ctl->tokens[0] = tok;
}

// Draft step (Algorithm 2 drafting, exit of Sec. 3.4): keep draft d, whose
// distribution's maximum was pmax; stop after it when pmax < gamma or the
// stage budget is reached, and set up the verification of [last, d_1..d_k].
__device__ inline void draft_commit(const HeadArgs &h, DevCtl *ctl, int d, float pmax) {
    DevState *st = h.st;
    const int j = st->k;
    st->drafts[j] = d;
    st->dpmax[j] = pmax;
    st->k = j + 1;
    st->n_draft_steps += 1;
    const bool exit_now = (pmax < st->gamma) || (j + 1 >= st->kcap);
    if (!exit_now) {
        ctl->pos = st->lc + j + 1;
        ctl->m_next = 1;
        ctl->tokens[0] = d;
    } else {
        st->phase = PHASE_VERIFY;
        ctl->pos = st->lc;
        ctl->m_next = j + 2;
        ctl->tokens[0] = st->last;
        for (int i = 0; i <= j; ++i)
            ctl->tokens[i + 1] = st->drafts[i];
    }
    post_mailbox(st, h.mb);
}

// End of a verification stage: the first n drafts are accepted and tok
// follows them.  The committed length advances past them, which rolls back
// the KV positions of rejected drafts; then the adaptive threshold update
// (Sec. 3.4, Eqs. 2-4), if on, and the set-up of the next stage.
__device__ inline void stage_commit(const HeadArgs &h, DevCtl *ctl, int n, int tok) {
    DevState *st = h.st;
    const int k = st->k;
    int e = st->emitted;
    for (int i = 0; i < n; ++i)
        h.out_tokens[e + i] = st->drafts[i];
    h.out_tokens[e + n] = tok;
    e += n + 1;
    st->emitted = e;
    if (h.stage_log && st->n_stages < h.stage_log_cap) {
        h.stage_log[2 * st->n_stages] = k;
        h.stage_log[2 * st->n_stages + 1] = n;
        h.gamma_log[st->n_stages] = st->gamma;
    }
    st->n_stages += 1;
    st->n_drafted += k;
    st->n_accepted += n;
    // Adaptive threshold: smooth the stage's acceptance rate into AR (the
    // first stage sets it), step the threshold up when AR is at most the
    // target and down otherwise, and smooth the step.  Float64, each
    // operation rounded on its own in the order of the equations
    // (contraction into FMAs is off, so the host-side definition gives the
    // same bits); a stage without drafts carries no acceptance rate and
    // leaves both unchanged.
    if (st->adaptive && k > 0) {
#pragma clang fp contract(off)
        const double ar_e = (double)n / (double)k;
        st->ar = st->n_updates == 0 ? ar_e : st->beta1 * st->ar + (1.0 - st->beta1) * ar_e;
        st->n_updates += 1;
        const double gt = st->ar <= st->alpha ? st->gamma_d + st->epsilon : st->gamma_d - st->epsilon;
        st->gamma_d = st->beta2 * st->gamma_d + (1.0 - st->beta2) * gt;
        st->gamma = __double2float_rn(st->gamma_d);
    }
    st->lc += n + 1;
    st->last = tok;
    if (e >= st->max_new) {
        st->gen_done = 1;
    } else {
        const int kcap = min(st->k_max, st->max_new - e - 1);
        st->k = 0;
        st->kcap = kcap;
        st->phase = kcap > 0 ? PHASE_DRAFT : PHASE_VERIFY;
    }
    ctl->pos = st->lc;
    ctl->m_next = 1;
    ctl->tokens[0] = st->last;
    post_mailbox(st, h.mb);
}

}  // namespace sdk
