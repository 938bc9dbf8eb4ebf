"""Drive the HIP path (through the C ABI) and the oracle on identical inputs, step
by step, and compare them.

Comparison rules (the GPU computes in fp32 with bf16 storage, the oracle in
fp32 with the same storage rounding):
  * logits: max |delta| <= tol over every verified / drafted row;
  * token decisions (prefill token, drafted tokens, target argmax through the
    accepted count and emitted tokens): identical wherever the oracle's top-2
    margin of the deciding row exceeds tol.  At a row whose margin is <= tol
    both choices are correct; the comparison of that slot stops there and the
    margin is reported.
"""
import numpy as np
import torch

from wf_fixtures import make_memory, make_prefix, plant_drafts
from oracle import OracleOpts, Target, Drafter, Session

from paper_2609_32869_amd import WhisperFlash, to_device_storage


def margin(row):
    top = np.partition(row.astype(np.float64), -2)[-2:]
    return float(top[1] - top[0])


def build_engine(cfg, W, max_batch):
    arrays = [W.values[name] for name, _ in W.order]
    return WhisperFlash.from_host(cfg, max_batch, arrays)


class Lockstep:
    """GPU engine over all prompts; the oracle follows the slots in ``check`` (all by
    default).  Slots are independent, so a sample of them checks the whole batch."""

    def __init__(self, cfg, W, prompts, max_new, tol, opts=None, mems=None, slots=None, check=None):
        self.cfg, self.W, self.tol = cfg, W, tol
        n = len(prompts)
        self.n = n
        self.eng = build_engine(cfg, W, n)
        if opts is None:
            opts = OracleOpts(dtype=np.float32, kv_bf16=(cfg.dtype == "bf16"), exact=cfg.d_model <= 384)
        self.T, self.D = Target(cfg, W.values, opts), Drafter(cfg, W.values, opts)
        slots = list(range(n)) if slots is None else slots
        if mems is None:
            mems = [make_memory(cfg, s) for s in slots]
        memt = torch.stack([to_device_storage(m, cfg.dtype) for m in mems])
        self.eng.encode_memory_set(0, memt)
        pmax = max(len(p) for p in prompts)
        toks = np.zeros((n, pmax), np.int32)
        for i, p in enumerate(prompts):
            toks[i, :len(p)] = p
        first = self.eng.prefill(0, torch.from_numpy(toks).cuda(), [len(p) for p in prompts], max_new)
        self.gpu_first = first.cpu().numpy()
        check = set(range(n) if check is None else check)
        self.sess = [Session(self.T, self.D, mems[i], prompts[i], max_new[i]) if i in check else None for i in range(n)]
        self.live = [i in check for i in range(n)]  # slot compared (until a near tie)
        self.near_ties = []             # (slot, what, margin)
        self.max_dlogit = 0.0
        self.max_tlogit = 0.0
        self.steps = 0
        self.accepted = []
        for i, s in enumerate(self.sess):
            if s is None:
                continue
            if self.gpu_first[i] != s.out[0]:
                m = margin(s.last_logits[-1])
                assert m <= tol, f"slot {i}: first token {self.gpu_first[i]} vs oracle {s.out[0]} (margin {m})"
                self.near_ties.append((i, "prefill", m))
                self.live[i] = False

    def step(self, k_max=8, override=None):
        """One wf_draft + wf_verify_accept on the GPU and the same round in the oracle."""
        cfg, tol, n = self.cfg, self.tol, self.n
        eng = self.eng
        eng.set_debug(True)
        drafts = eng.draft(0, n)
        torch.cuda.synchronize()
        dg = drafts.cpu().numpy()
        dlog = eng.draft_logits()[:n, 1:].cpu().numpy()
        used = dg.copy() if override is None else np.asarray(override, np.int32).copy()
        for i, s in enumerate(self.sess):
            if not self.live[i] or s.done:
                continue
            ol = s.draft_logits()
            self.max_dlogit = max(self.max_dlogit, float(np.abs(ol - dlog[i]).max()))
            assert np.abs(ol - dlog[i]).max() <= tol, f"slot {i}: draft logits differ by {np.abs(ol - dlog[i]).max()}"
            for j in range(cfg.block_k):
                oj = int(np.argmax(ol[j]))
                if oj != dg[i, j]:
                    m = margin(ol[j])
                    assert m <= tol, f"slot {i}: draft token {j}: {dg[i, j]} vs {oj} (margin {m})"
        out, n_out, n_acc, done = eng.verify_accept(0, torch.from_numpy(used).cuda(), k_max)
        torch.cuda.synchronize()
        out, n_out, n_acc, done = (t.cpu().numpy() for t in (out, n_out, n_acc, done))
        tlog = eng.target_logits()[:n].cpu().numpy()
        for i, s in enumerate(self.sess):
            if not self.live[i]:
                continue
            if s.done:
                assert n_out[i] == 0 and done[i] == 1
                continue
            rec = s.verify_accept(used[i], k_max)
            k = rec["k"]
            ol = s.last_logits
            d = float(np.abs(ol - tlog[i, :k + 1]).max())
            self.max_tlogit = max(self.max_tlogit, d)
            assert d <= tol, f"slot {i}: target logits differ by {d}"
            gpu_tokens = list(out[i, :n_out[i]])
            if gpu_tokens != rec["tokens"] or n_acc[i] != rec["a"]:
                # find the deciding row: first row whose argmax differs between the two
                rows = [r for r in range(k + 1) if int(np.argmax(ol[r])) != int(np.argmax(tlog[i, r]))]
                assert rows, f"slot {i}: tokens differ without an argmax difference"
                m = margin(ol[rows[0]])
                assert m <= tol, f"slot {i}: tokens {gpu_tokens} vs {rec['tokens']} (margin {m})"
                self.near_ties.append((i, f"step {self.steps} row {rows[0]}", m))
                self.live[i] = False
                continue
            assert bool(done[i]) == s.done
            self.accepted.append(int(n_acc[i]))
        self.steps += 1
        return out, n_out, n_acc, done

    def verify_only(self, k_max=0, override=None):
        """One wf_verify_accept with no draft call before it (the oracle likewise):
        the drafter history must still receive the verified rows."""
        cfg, tol, n = self.cfg, self.tol, self.n
        eng = self.eng
        eng.set_debug(True)
        used = np.zeros((n, cfg.block_k), np.int32) if override is None else np.asarray(override, np.int32).copy()
        out, n_out, n_acc, done = eng.verify_accept(0, torch.from_numpy(used).cuda(), k_max)
        torch.cuda.synchronize()
        out, n_out, n_acc, done = (t.cpu().numpy() for t in (out, n_out, n_acc, done))
        tlog = eng.target_logits()[:n].cpu().numpy()
        for i, s in enumerate(self.sess):
            if not self.live[i] or s.done:
                continue
            rec = s.verify_accept(used[i], k_max)
            k = rec["k"]
            d = float(np.abs(s.last_logits - tlog[i, :k + 1]).max())
            self.max_tlogit = max(self.max_tlogit, d)
            assert d <= tol, f"slot {i}: target logits differ by {d}"
            if list(out[i, :n_out[i]]) != rec["tokens"]:
                m = margin(s.last_logits[0])
                assert m <= tol, f"slot {i}: tokens {list(out[i, :n_out[i]])} vs {rec['tokens']} (margin {m})"
                self.near_ties.append((i, f"verify {self.steps}", m))
                self.live[i] = False
        self.steps += 1

    def graph_step(self, override, outs, ovr_dev, k_max=8):
        """One graph-replayed wf_step (the path the benchmark times) with planted
        drafts; the drafter runs inside the step and its logits are compared too."""
        cfg, tol, n = self.cfg, self.tol, self.n
        eng = self.eng
        ovr_dev.copy_(torch.from_numpy(np.asarray(override, np.int32)))
        eng.step(0, n, k_max, draft_override=ovr_dev, outs=outs, use_graph=True)
        torch.cuda.synchronize()
        out, n_out, n_acc, done = (t.cpu().numpy() for t in outs)
        dg = eng.last_draft()[:n].cpu().numpy()
        dlog = eng.draft_logits()[:n, 1:].cpu().numpy()
        tlog = eng.target_logits()[:n].cpu().numpy()
        for i, s in enumerate(self.sess):
            if not self.live[i]:
                continue
            if s.done:
                assert n_out[i] == 0 and done[i] == 1
                continue
            ol = s.draft_logits()
            dd = float(np.abs(ol - dlog[i]).max())
            self.max_dlogit = max(self.max_dlogit, dd)
            assert dd <= tol, f"slot {i}: draft logits differ by {dd}"
            for j in range(cfg.block_k):
                oj = int(np.argmax(ol[j]))
                if oj != dg[i, j]:
                    m = margin(ol[j])
                    assert m <= tol, f"slot {i}: draft token {j}: {dg[i, j]} vs {oj} (margin {m})"
            rec = s.verify_accept(override[i], k_max)
            k = rec["k"]
            d = float(np.abs(s.last_logits - tlog[i, :k + 1]).max())
            self.max_tlogit = max(self.max_tlogit, d)
            assert d <= tol, f"slot {i}: target logits differ by {d}"
            gpu_tokens = list(out[i, :n_out[i]])
            if gpu_tokens != rec["tokens"] or n_acc[i] != rec["a"]:
                rows = [r for r in range(k + 1) if int(np.argmax(s.last_logits[r])) != int(np.argmax(tlog[i, r]))]
                assert rows, f"slot {i}: tokens differ without an argmax difference"
                m = margin(s.last_logits[rows[0]])
                assert m <= tol, f"slot {i}: tokens {gpu_tokens} vs {rec['tokens']} (margin {m})"
                self.near_ties.append((i, f"step {self.steps} row {rows[0]}", m))
                self.live[i] = False
                continue
            assert bool(done[i]) == s.done
            self.accepted.append(int(n_acc[i]))
        self.steps += 1
        return out, n_out, n_acc, done

    def close(self):
        self.eng.close()
