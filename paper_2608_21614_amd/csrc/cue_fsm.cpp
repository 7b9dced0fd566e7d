// cue_fsm.cpp -- stage-boundary detection over generated token streams (SAEM
// Section IV-B.1, "sliding-window pattern matching"): after every decode step the
// newest token of each sequence is fed to a finite-state machine that tracks the
// partial matches of every transition cue, so a cue that spans several subword
// tokens is recognised the step its last token is generated.
//
// The machine is a multi-pattern automaton over token ids (Aho-Corasick): a trie
// of the cues, a failure link per state (the state of the longest proper suffix
// of its token string that is also a cue prefix) and, per state, the longest cue
// that ends there.  Its state is equivalent to a window of the last
// (longest cue - 1) tokens, at one int32 per sequence.  Host code only.
//
// Serialized form (int32 words, caller-owned):
//   [0] magic, [1] states S, [2] edges S-1, [3] cues
//   edge_begin [S+1]   edges of state s are edge_begin[s] .. edge_begin[s+1]-1
//   fail [S], out [S]  failure link; id of the longest cue ending in s, or -1
//   edge_tok [S-1], edge_next [S-1]   sorted by token within each state
#include <stdint.h>

#include <algorithm>
#include <deque>
#include <utility>
#include <vector>

#include "saem_moe.h"

namespace {

constexpr int32_t kMagic = 0x43554546;  // "CUEF"

int64_t words_for_states(int64_t states) { return 4 + (states + 1) + 2 * states + 2 * (states - 1); }

struct View {
    int32_t S = 0, E = 0, ncues = 0;
    const int32_t* begin = nullptr;
    const int32_t* fail = nullptr;
    const int32_t* out = nullptr;
    const int32_t* tok = nullptr;
    const int32_t* nxt = nullptr;
};

bool view_of(const int32_t* f, View* v) {
    if (!f || f[0] != kMagic || f[1] < 1 || f[2] != f[1] - 1 || f[3] < 0) return false;
    v->S = f[1];
    v->E = f[2];
    v->ncues = f[3];
    v->begin = f + 4;
    v->fail = v->begin + v->S + 1;
    v->out = v->fail + v->S;
    v->tok = v->out + v->S;
    v->nxt = v->tok + v->E;
    return true;
}

// child of state s on token t, or -1
int32_t child(const View& v, int32_t s, int32_t t) {
    const int32_t* lo = v.tok + v.begin[s];
    const int32_t* hi = v.tok + v.begin[s + 1];
    const int32_t* p = std::lower_bound(lo, hi, t);
    return (p != hi && *p == t) ? v.nxt[p - v.tok] : -1;
}

}  // namespace

extern "C" {

int64_t moe_cue_fsm_words(int64_t total_tokens) {
    if (total_tokens < 0) return -1;
    return words_for_states(total_tokens + 1);
}

moe_status moe_cue_build(int32_t n_cues, const int32_t* cue_offsets, const int32_t* cue_tokens, int32_t* fsm,
                         int64_t fsm_words) {
    if (n_cues < 0 || !fsm || (n_cues > 0 && (!cue_offsets || !cue_tokens))) return MOE_ERR_INVALID_ARG;
    int64_t total = 0;
    if (n_cues > 0) {
        if (cue_offsets[0] != 0) return MOE_ERR_INVALID_ARG;
        for (int32_t c = 0; c < n_cues; ++c) {
            if (cue_offsets[c + 1] <= cue_offsets[c]) return MOE_ERR_INVALID_ARG;  // every cue has a token
        }
        total = cue_offsets[n_cues];
        for (int64_t i = 0; i < total; ++i)
            if (cue_tokens[i] < 0) return MOE_ERR_INVALID_ARG;
    }
    if (fsm_words < moe_cue_fsm_words(total)) return MOE_ERR_WORKSPACE;

    // trie: children kept sorted by token
    std::vector<std::vector<std::pair<int32_t, int32_t>>> kids(1);
    std::vector<int32_t> out(1, -1), depth(1, 0);
    for (int32_t c = 0; c < n_cues; ++c) {
        int32_t s = 0;
        for (int32_t i = cue_offsets[c]; i < cue_offsets[c + 1]; ++i) {
            const int32_t t = cue_tokens[i];
            auto& ks = kids[s];
            auto it = std::lower_bound(ks.begin(), ks.end(), std::make_pair(t, INT32_MIN));
            if (it != ks.end() && it->first == t) {
                s = it->second;
            } else {
                const int32_t ns = (int32_t)kids.size();
                ks.insert(it, {t, ns});
                kids.emplace_back();
                out.push_back(-1);
                depth.push_back(depth[s] + 1);
                s = ns;
            }
        }
        if (out[s] < 0) out[s] = c;  // a repeated cue keeps its lowest id
    }
    const int32_t S = (int32_t)kids.size();

    // failure links breadth first; out[s] becomes the longest cue ending in s:
    // s's own cue if it is one (the deepest), else the one of its failure state
    std::vector<int32_t> fail(S, 0);
    std::deque<int32_t> q;
    for (const auto& kv : kids[0]) q.push_back(kv.second);
    while (!q.empty()) {
        const int32_t s = q.front();
        q.pop_front();
        if (out[s] < 0) out[s] = out[fail[s]];
        for (const auto& kv : kids[s]) {
            int32_t f = fail[s];
            int32_t g = -1;
            for (;;) {
                auto& fk = kids[f];
                auto it = std::lower_bound(fk.begin(), fk.end(), std::make_pair(kv.first, INT32_MIN));
                if (it != fk.end() && it->first == kv.first && it->second != kv.second) {
                    g = it->second;
                    break;
                }
                if (f == 0) break;
                f = fail[f];
            }
            fail[kv.second] = g < 0 ? 0 : g;
            q.push_back(kv.second);
        }
    }

    fsm[0] = kMagic;
    fsm[1] = S;
    fsm[2] = S - 1;
    fsm[3] = n_cues;
    int32_t* begin = fsm + 4;
    int32_t* fl = begin + S + 1;
    int32_t* ou = fl + S;
    int32_t* tok = ou + S;
    int32_t* nxt = tok + (S - 1);
    int32_t e = 0;
    for (int32_t s = 0; s < S; ++s) {
        begin[s] = e;
        fl[s] = fail[s];
        ou[s] = out[s];
        for (const auto& kv : kids[s]) {
            tok[e] = kv.first;
            nxt[e] = kv.second;
            ++e;
        }
    }
    begin[S] = e;
    return MOE_OK;
}

moe_status moe_cue_step(const int32_t* fsm, int32_t batch, const int32_t* tokens, int32_t* state,
                        int32_t* matched) {
    View v;
    if (!view_of(fsm, &v) || batch < 0 || (batch > 0 && (!tokens || !state || !matched)))
        return MOE_ERR_INVALID_ARG;
    for (int32_t b = 0; b < batch; ++b)
        if (state[b] < 0 || state[b] >= v.S) return MOE_ERR_INVALID_ARG;
    for (int32_t b = 0; b < batch; ++b) {
        const int32_t t = tokens[b];
        if (t < 0) {  // no token this step (an idle or finished sequence): the window restarts
            state[b] = 0;
            matched[b] = -1;
            continue;
        }
        int32_t s = state[b];
        int32_t n = child(v, s, t);
        while (n < 0 && s != 0) {
            s = v.fail[s];
            n = child(v, s, t);
        }
        s = n < 0 ? 0 : n;
        state[b] = s;
        matched[b] = v.out[s];
    }
    return MOE_OK;
}

}  // extern "C"
