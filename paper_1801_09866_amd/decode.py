"""Closing the decode loop on the device.

After a frame, the decoder extends some hypotheses by a word: the history
of an extended hypothesis is the GRU output h' that the library has just
produced for its parent (Sec. 2.4: the outputs become the next histories).
Here those histories never leave HBM and are never copied: each frame passes
`hist_ptr`, the device addresses of its histories' rows, which point into
the h' outputs of earlier frames (or into the initial histories).

The beam's evolution comes from a seeded plan (workload.decode_plan) that
does not look at scores, so any implementation that follows the same plan
meets the same keys.
"""
from __future__ import annotations

import numpy as np
import torch


class DeviceDecodeLoop:
    """Runs a decode plan through a Scorer with history handles.

    init_vec: device tensor [beam, L*H] fp32, the histories of frame 0.
    Every frame's outputs (scores, h', statuses) stay alive on the device for
    as long as this object does, since later frames may point at them.
    """

    def __init__(self, scorer, init_vec):
        self.sc = scorer
        self.dev = init_vec.device
        self.row_bytes = init_vec.shape[1] * init_vec.element_size()
        self.init = init_vec
        self.outs = []

    def run(self, plan, debug=True):
        src = [self.init.data_ptr() + j * self.row_bytes for j in range(len(plan[0].words))]
        for t, fr in enumerate(plan):
            if t > 0:
                base = self.outs[-1]["hnew"].data_ptr()
                src = [base + int(p) * self.row_bytes if adv else src[int(p)]
                       for p, adv in zip(fr.prev, fr.advanced)]
            hp = torch.tensor(src, dtype=torch.int64).to(self.dev, non_blocking=False)
            d = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(self.dev)
            out = self.sc.score_frame(None, d(fr.words), d(fr.q_hist), d(fr.q_tgt), hist_ptr=hp, debug=debug)
            out["hist_ptr"] = hp   # keeps the handle array alive while the frame runs
            self.outs.append(out)
        return self.outs
