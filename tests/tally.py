"""Registry of parity tallies: every GPU-versus-oracle case records how many
comparisons matched exactly and how many differed at an excused near-tie
decision, per stage; tests/conftest.py prints them at the end of the run so
that a quiet (-q) log still shows them."""

REGISTRY = []


class Tally:
    STAGES = ("plan", "replay", "verify")

    def __init__(self, name, register=True):
        self.name = name
        self.exact = {s: 0 for s in self.STAGES}
        self.flagged_by = {s: 0 for s in self.STAGES}
        self.notes = []
        self.request_steps = 0
        self.steps = 0
        self.max_lse_err = 0.0
        if register:
            REGISTRY.append(self)

    def ok(self, stage):
        self.exact[stage] += 1

    def flag(self, stage, what):
        self.flagged_by[stage] += 1
        self.notes.append(what)

    @property
    def flagged(self):
        return sum(self.flagged_by.values())

    @property
    def total_exact(self):
        return sum(self.exact.values())

    def line(self):
        e, f = self.exact, self.flagged_by
        return ("%-40s rounds %4d req-steps %5d | plan %5d/%d | replay %6d/%d | verify %5d/%d | max|dlse_t| %.1e%s"
                % (self.name, self.steps, self.request_steps, e["plan"], f["plan"], e["replay"], f["replay"],
                   e["verify"], f["verify"], self.max_lse_err, ("  " + "; ".join(self.notes[:3])) if self.notes else ""))
