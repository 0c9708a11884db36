"""Readers for the hand-worked text fixtures in this folder."""
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def _lines(name):
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                yield line.split()


def gae_example():
    params, rows = {}, []
    for tok in _lines("skip_observation_gae_example.txt"):
        if tok[0] in ("gamma", "lambda"):
            params[tok[0]] = float(tok[1])
        elif tok[0] == "cu_seqlens":
            params["cu"] = np.array([int(x) for x in tok[1:]], np.int32)
        else:
            rows.append([float(x) for x in tok])
    a = np.array(rows)
    return dict(gamma=params["gamma"], lam=params["lambda"], cu=params["cu"],
                mask=a[:, 1].astype(np.uint8), values=a[:, 2].astype(np.float32),
                rewards=a[:, 3].astype(np.float32), adv=a[:, 4], ret=a[:, 5])


def dis_example():
    d, rows = {"loss": np.zeros(2)}, []
    for tok in _lines("dis_loss_example.txt"):
        if tok[0] in ("eps_low", "eps_high"):
            d[tok[0]] = float(tok[1])
        elif tok[0] == "loss":
            d["loss"][int(tok[1])] = float(tok[2])
        elif tok[0] == "counts":
            d["counts"] = np.array([int(x) for x in tok[1:]], np.int64)
        else:
            rows.append([float(x) for x in tok])
    a = np.array(rows)
    d.update(mask=a[:, 1].astype(np.uint8), logp=a[:, 2].astype(np.float32),
             logp_rollout=a[:, 3].astype(np.float32), adv=a[:, 4].astype(np.float32),
             flags=a[:, 5].astype(np.uint8), g=a[:, 6])
    return d
