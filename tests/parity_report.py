"""Lines the parity tests record for the end-of-run summary (the error figures
of every full-size comparison with the oracle stay visible in the run's tail,
where captured output would hide them)."""

LINES = []


def record(line: str) -> None:
    LINES.append(line)
