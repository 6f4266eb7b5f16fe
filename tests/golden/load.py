"""Readers for the text fixtures in this directory."""
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))


def table(name):
    rows = []
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.split("#", 1)[0].strip()
            if line:
                rows.append([float(t) for t in line.split()])
    return np.array(rows)
