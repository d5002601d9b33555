"""The library workspace under graph capture, in a fresh process (so that the
workspace starts empty): a captured round keeps working after a larger eager
call has grown the workspace (the buffer the graph holds is retired, never
freed), and a call that would have to grow the workspace while its stream is
captured returns SQ_ERR_CAPTURE and enqueues nothing."""
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

CHILD = r'''
import sys
sys.path.insert(0, sys.argv[1])
import torch
import paper_2609_21704_amd as sq
from paper_2609_21704_amd import synth
from paper_2609_21704_amd.configs import CONFIGS
from paper_2609_21704_amd.rounds import Round, Stack, round_uniforms

dev = torch.device("cuda:0")
torch.cuda.set_device(dev)
cfg = CONFIGS[0]
rnd = Round(Stack(cfg, dev), temperature=1.0)
ud, ua = round_uniforms(cfg, 2, dev)
rnd.set_uniforms(ud[0], ua[0])
rnd.capture()                      # one eager round (the workspace is allocated), then the graph
b = rnd.buf

def state():
    return [t.clone() for t in (b.draft_logits, b.target_logits, b.draft_tokens, b.n_accepted, b.next_token)]

def same(x, y):
    return all(torch.equal(p, q) for p, q in zip(x, y))

rnd.set_uniforms(ud[1], ua[1])
rnd.run()
torch.cuda.synchronize()
eager = state()
rnd.replay()
torch.cuda.synchronize()
assert same(state(), eager), "replay before growth"
print("step: replay matches the eager round", flush=True)

# a larger eager call: 200000 one-token rows need ~14 MB of accept scratch,
# more than the round's, so the workspace grows (the round's buffer is retired)
big = 200000
tgt = synth.normal_f32((big, 1, 1), 1.0, 5, dev)
u = synth.uniform_u24((big, 1), 6, dev)
n, t = sq.sq_spec_accept(None, tgt, None, u, 1.0)
torch.cuda.synchronize()
assert bool((t == 0).all()) and bool((n == 0).all())
for _ in range(3):
    rnd.replay()
    torch.cuda.synchronize()
    assert same(state(), eager), "replay after growth"
rnd.run()
torch.cuda.synchronize()
assert same(state(), eager), "eager round after growth"
print("step: replays after the workspace grew match the eager round", flush=True)

# growth needed while the stream is captured: refused with SQ_ERR_CAPTURE
huge = 2000000
tgt2 = synth.normal_f32((huge, 1, 1), 1.0, 7, dev)
u2 = synth.uniform_u24((huge, 1), 8, dev)
status = None
g = torch.cuda.CUDAGraph()
try:
    with torch.cuda.graph(g):
        try:
            sq.sq_spec_accept(None, tgt2, None, u2, 1.0)
        except sq.SpecQuantError as e:
            status = e.status
except Exception as e:  # ending the empty capture is not under test
    print("capture end:", type(e).__name__, flush=True)
assert status == 8, status
torch.cuda.synchronize()
rnd.replay()
torch.cuda.synchronize()
assert same(state(), eager), "replay after the refused call"
n2, t2 = sq.sq_spec_accept(None, tgt2, None, u2, 1.0)   # outside capture the same call grows and runs
torch.cuda.synchronize()
assert bool((t2 == 0).all())
print("CAPTURE_OK", flush=True)
'''


def test_workspace_growth_and_capture_in_a_fresh_process():
    print("child: capture / workspace growth at workload 0", flush=True)
    res = subprocess.run([sys.executable, "-c", CHILD, ROOT], capture_output=True, text=True, timeout=300)
    print(res.stdout[-2000:], res.stderr[-2000:])
    assert res.returncode == 0 and "CAPTURE_OK" in res.stdout
