"""Plain oracle of paired co-scheduling (host scheduling policy).

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle``: only the test suite may
import it.  Pure Python over small request streams; it shares no code with the
library's scheduler.

What it follows (Sec. 2.4, CFG via paired request co-scheduling):
  * a request with a CFG scale w > 1 is served as its Main request plus an
    auto-allocated Companion request with a null prompt;
  * the two are one scheduling unit: admitted together, always run in the same
    step, retired together;
  * a step's token budget is split equally between the two members of a pair.
And from Sec. 3.4: guidance is applied only in the short audio phase, so the
Companion takes part only there (text comes first, as in the mixed models of
Sec. 2.3, and its tokens are greedy and unmerged).

Readings where the paper is silent (each also listed in the design notes):
  * a step first gives one token to every decoding row, then prompt chunks to
    units still prefilling, oldest first, then admits waiting units strictly in
    arrival order while rows and tokens remain (the first that does not fit
    stops admission);
  * "split equally": both members of a pair are granted the same count
    c = min(floor(tokens left / 2), the larger of their remaining prompts) and
    the pair is charged 2c; a member uses at most its own remainder;
  * a unit decodes from the step after its last prompt token; decode step t
    < text_len is a text step (Main only), then n_frames + drain audio steps
    (Main and Companion for a pair, at audio step t - text_len);
  * the Companion joins the audio phase with a copy of the Main sequence (a
    prefix-cache hit, no prompt tokens); its context is its null prompt plus
    the t tokens the pair has decoded;
  * rows are slots of the batch, the lowest free ones, held from admission to
    retirement.

parity pinned by: a step-by-step trace worked by hand from the rules above,
and invariants over random streams (budget, equal grants, pairs together,
arrival order, every token accounted for).
"""
from __future__ import annotations

ROW_COND, ROW_UNCOND, ROW_SOLO, ROW_TEXT = 0, 1, 2, 3


class CoScheduler:
    def __init__(self, max_rows, token_budget, null_prompt_len, drain_steps):
        assert max_rows >= 1 and token_budget >= max_rows
        assert null_prompt_len >= 1 and drain_steps >= 0
        self.max_rows = max_rows
        self.budget = token_budget
        self.null_prompt = null_prompt_len
        self.drain = drain_steps
        self.queue = []          # requests in arrival order (waiting and running)
        self.free = [True] * max_rows
        self.count = 0

    def submit(self, cfg_w, prompt_len, text_len, n_frames):
        pair = cfg_w > 1.0
        members = ["main", "comp"] if pair else ["main"]
        req = {
            "id": self.count, "w": cfg_w, "pair": pair, "members": members,
            "prompt": prompt_len, "text": text_len, "frames": n_frames,
            "state": "waiting", "t": 0,
            "todo": {"main": prompt_len, "comp": self.null_prompt if pair else 0},
            "fed": {"main": 0, "comp": 0},
            "slot": {},
        }
        self.count += 1
        self.queue.append(req)
        return req["id"]

    def _grant(self, req, tokens):
        """Prompt tokens of each member this step, and the tokens charged."""
        if req["pair"]:
            c = min(tokens // 2, max(req["todo"]["main"], req["todo"]["comp"]))
            return {"main": min(c, req["todo"]["main"]), "comp": min(c, req["todo"]["comp"])}, 2 * c
        c = min(tokens, req["todo"]["main"])
        return {"main": c}, c

    def step(self):
        """Plan and apply one step.  Returns (rows, head, finished): rows are
        (id, member, tokens, context) of the backbone batch, head rows are
        (id, member, row kind, step, partner head index, grid slot)."""
        tokens = self.budget
        decoding = [q for q in self.queue if q["state"] == "decode"]
        for q in decoding:
            in_audio = q["t"] >= q["text"]
            tokens -= 2 if (in_audio and q["pair"]) else 1
        grants = {}
        for q in self.queue:
            if q["state"] == "prefill":
                grants[q["id"]], charged = self._grant(q, tokens)
                tokens -= charged
        for q in self.queue:
            if q["state"] != "waiting":
                continue
            need = len(q["members"])
            if sum(self.free) < need or tokens < need:
                break
            for m in q["members"]:
                s = self.free.index(True)
                self.free[s] = False
                q["slot"][m] = s
            q["state"] = "prefill"
            grants[q["id"]], charged = self._grant(q, tokens)
            tokens -= charged
        assert tokens >= 0

        rows, head = [], []
        for q in self.queue:
            if q["state"] == "decode":
                t = q["t"]
                if t < q["text"]:
                    rows.append((q["id"], 0, 1, q["prompt"] + t))
                    head.append((q["id"], 0, ROW_TEXT, t, -1, -1))
                elif not q["pair"]:
                    rows.append((q["id"], 0, 1, q["prompt"] + t))
                    head.append((q["id"], 0, ROW_SOLO, t - q["text"], -1, q["slot"]["main"]))
                else:
                    h = len(head)
                    rows.append((q["id"], 0, 1, q["prompt"] + t))
                    head.append((q["id"], 0, ROW_COND, t - q["text"], h + 1, q["slot"]["main"]))
                    rows.append((q["id"], 1, 1, self.null_prompt + t))
                    head.append((q["id"], 1, ROW_UNCOND, t - q["text"], h, -1))
            elif q["state"] == "prefill":
                for k, m in enumerate(q["members"]):
                    g = grants[q["id"]][m]
                    if g > 0:
                        rows.append((q["id"], k, g, q["fed"][m]))

        finished = []
        for q in list(self.queue):
            if q["state"] == "decode":
                q["t"] += 1
                if q["t"] == q["text"] + q["frames"] + self.drain:
                    for s in q["slot"].values():
                        self.free[s] = True
                    finished.append(q["id"])
                    self.queue.remove(q)
            elif q["state"] == "prefill":
                for m, g in grants[q["id"]].items():
                    q["todo"][m] -= g
                    q["fed"][m] += g
                if all(v == 0 for v in q["todo"].values()):
                    q["state"] = "decode"
        return rows, head, finished
