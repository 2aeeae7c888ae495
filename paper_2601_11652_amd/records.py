"""The command line that a measurement record was made with, stored in the record itself."""
from __future__ import annotations

import shlex
import sys


def command_line(module: str | None, argv=None) -> str:
    """`python -m module args...` (or `python script args...` when module is None) for the
    arguments of this run: argv if given, else the process's own."""
    args = list(sys.argv[1:] if argv is None else argv)
    head = ["python", "-m", module] if module else ["python", sys.argv[0]]
    return " ".join(shlex.quote(a) for a in head + [str(a) for a in args])
