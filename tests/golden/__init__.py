"""Text fixtures transcribed from the paper's tables; each file names the table it comes from."""
import os

HERE = os.path.dirname(os.path.abspath(__file__))


def load(name: str):
    rows = []
    with open(os.path.join(HERE, name)) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            rows.append([float(x) if "." in x else int(x) for x in line.split()])
    return rows
